// HIP kernels of the KV-cache splice for gfx950 (MI355X), and the C-ABI entry points that
// enqueue them.
//
// The path is bandwidth-bound element movement with a little fp32 arithmetic on the rotary
// band (about 0.1-0.4 flop per byte), so there is no matrix-core work here: rows are moved as
// 16-byte vectors, and the re-anchoring rotation (Eq. "rotate": each pair (a, b) becomes
// (a c - b s, a s + b c)) is applied in registers between the load and the store of a moved
// row, with the result rounded to bf16 by the hardware's round-to-nearest-even conversion.
// cos/sin of (shift * theta_i) come from the host, evaluated in fp64 once per call and shift,
// travel in the kernel arguments (or the call's workspace) and are staged once per workgroup in
// LDS.
//
// Access shape.  The 16-byte chunks of the moved rows are laid end to end over the threads, so
// that every load and store instruction of a 64-wide wavefront covers about 1 KiB of whole rows
// (a thread repeats its chunk position in a few rows or layers: two consecutive rows of a
// rotating round item and one row of a copy in the round kernel, two layers in the paged
// kernels, eight strided chunks in a tile); that is the shape that streams near the copy ceiling
// of the chip.  For a half-split (NEOX) band the partner half of a chunk lives in another lane of
// the same wavefront and is exchanged with a lane shuffle instead of being loaded twice.  Index
// arithmetic uses precomputed multiply-shift division.
//
// In-place contiguous compaction.  A segment moved left by m rows writes row x with the old
// content of row x + m.  The host splits the segment into equal rounds of at most m rows taken
// in ascending order (descending for a right shift): inside a round sources and destinations
// are disjoint, and every row a round overwrites was read by an earlier round, so consecutive
// launches on one stream order the whole move.  When some shift of a call is too small for a
// few large rounds, the whole call (every move and replacement copy) runs as ordered tiles:
// workgroups take tickets in start order and wait on per-tile "source read" flags, so that no
// tile overwrites rows another tile has still to read (contig_tile_kernel).  Layouts whose
// half-split partners cannot be exchanged between lanes use ordered chains instead: chain c owns
// rows c, c+m, c+2m, ... and one thread walks it in order, overwriting only rows it has already
// read itself.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <vector>

#include "kparams.hpp"
#include "leyline.h"
#include "plan.hpp"

namespace leyline {

// Launch shape and streaming hints (compile-time constants; the defaults are the tuned ones).
#ifndef LEYLINE_TPB
#define LEYLINE_TPB 512
#endif
#ifndef LEYLINE_WIN
#define LEYLINE_WIN 8
#endif
#ifndef LEYLINE_NT_LOAD
#define LEYLINE_NT_LOAD 1
#endif
#ifndef LEYLINE_NT_STORE
#define LEYLINE_NT_STORE 1
#endif

constexpr int TPB = LEYLINE_TPB;
#ifndef LEYLINE_CONTIG_RPT
#define LEYLINE_CONTIG_RPT 2
#endif
#ifndef LEYLINE_MOVE_TPB
#define LEYLINE_MOVE_TPB 256
#endif
constexpr int CRPT = LEYLINE_CONTIG_RPT;   // rows per thread of a rotating round item
// Rows per thread of a round-kernel item: CRPT when it rotates; with fp32 pairs one when it only
// copies (a V plane, a replacement copy), with fp64 pairs CRPT as well (there the rotating
// workgroups are bound by their pair arithmetic, and the GQA splice runs 4 points slower with
// one-row copies beside them).  The kernel and the launcher's grid both take it from here.
LEYLINE_HD inline int round_rows_per_thread(bool rotates) { return rotates || LEYLINE_PAIR_F64 ? CRPT : 1; }
constexpr int MOVE_TPB = LEYLINE_MOVE_TPB; // its workgroup size
#ifndef LEYLINE_PAGED_TPB
#define LEYLINE_PAGED_TPB 256
#endif
#ifndef LEYLINE_GATHER_SPLIT_PAGE
#define LEYLINE_GATHER_SPLIT_PAGE 4    // smallest page size whose gather is split by XCD
#endif
#ifndef LEYLINE_PAGED_LPT
#define LEYLINE_PAGED_LPT 2
#endif
constexpr int PAGED_TPB = LEYLINE_PAGED_TPB;   // paged gather workgroup size
constexpr int PAGED_LPT = LEYLINE_PAGED_LPT;   // layers per paged-gather thread
constexpr int WIN = LEYLINE_WIN;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// 16-byte vector accesses.  Moved rows and rotated bands are touched exactly once per call, so
// the streaming (nontemporal) forms keep them from displacing other data in the caches.
__device__ __forceinline__ u32x4 ld16(const char* p) {
#if LEYLINE_NT_LOAD
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
#else
    return *reinterpret_cast<const u32x4*>(p);
#endif
}
__device__ __forceinline__ void st16(char* p, u32x4 v) {
#if LEYLINE_NT_STORE
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
#else
    *reinterpret_cast<u32x4*>(p) = v;
#endif
}


// ----------------------------------------------------------------------- element helpers ---

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 values -> two bf16 in one word (low half = a), round to nearest even.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    const bf16x2 v = __builtin_convertvector(f32x2{a, b}, bf16x2);
    return __builtin_bit_cast(uint32_t, v);
}

// (a, b) -> (a c - b s, a s + b c) (Eq. "rotate").  BF16: the results are bf16-bound, and come back
// as floats whose nearest-even bf16 is the stored value.  With fp64 pairs the products are fp64
// and each result is rounded once (to odd for bf16, see f32_round_odd; to nearest-even for fp32).
// fp64 pairs are computed without fused multiply-adds, as two rounded products and a rounded sum
// (the plain evaluation of the formula): a fused form rounds differently in the last place, and
// that can move a near-cancelling result across a rounding boundary of the storage type.
template <bool BF16>
__device__ __forceinline__ void rot_pair(float& a, float& b, const KCosSin& k) {
#if LEYLINE_PAIR_F64
#pragma clang fp contract(off)
    const double x = a, y = b;
    const double a2 = x * k.c - y * k.s;
    const double b2 = x * k.s + y * k.c;
    a = BF16 ? f32_round_odd(a2) : float(a2);
    b = BF16 ? f32_round_odd(b2) : float(b2);
#else
    const float a2 = a * k.c - b * k.s;
    const float b2 = a * k.s + b * k.c;
    a = a2;
    b = b2;
#endif
}

// One member of a half-split pair, on the lane that holds it: the low member a becomes
// a c - b s, the high member b becomes b c + a s, i.e. mine * c + partner * (lo ? -s : s).
template <bool BF16>
__device__ __forceinline__ float rot_own(float mine, float partner, const KCosSin& k, bool lo) {
#if LEYLINE_PAIR_F64
#pragma clang fp contract(off)
    const double r = double(mine) * k.c + double(partner) * (lo ? -k.s : k.s);
    return BF16 ? f32_round_odd(r) : float(r);
#else
    return mine * k.c + partner * (lo ? -k.s : k.s);
#endif
}

template <int ESZ> struct Elt { static constexpr int EPC = 16 / ESZ; };   // elements per chunk

// Interleaved chunk: EPC/2 pairs (2i, 2i+1), cos/sin from table[cs + i].
template <int ESZ> __device__ __forceinline__ void rot_interleaved(u32x4& v, const KCosSin* t, int32_t cs);
template <> __device__ __forceinline__ void rot_interleaved<2>(u32x4& v, const KCosSin* t, int32_t cs) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const KCosSin k = t[cs + i];
        float a = bf_lo(v[i]), b = bf_hi(v[i]);
        rot_pair<true>(a, b, k);
        v[i] = pack_bf16(a, b);
    }
}
template <> __device__ __forceinline__ void rot_interleaved<4>(u32x4& v, const KCosSin* t, int32_t cs) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const KCosSin k = t[cs + i];
        float a = __uint_as_float(v[2 * i]), b = __uint_as_float(v[2 * i + 1]);
        rot_pair<false>(a, b, k);
        v[2 * i] = __float_as_uint(a);
        v[2 * i + 1] = __float_as_uint(b);
    }
}

// Half-split chunks: element e of the low-half chunk `x` pairs with element e of the high-half
// chunk `y`; EPC pairs with cos/sin table[cs + e].  Both chunks are updated.
template <int ESZ> __device__ __forceinline__ void rot_halves(u32x4& x, u32x4& y, const KCosSin* t, int32_t cs);
template <> __device__ __forceinline__ void rot_halves<2>(u32x4& x, u32x4& y, const KCosSin* t, int32_t cs) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const KCosSin k0 = t[cs + 2 * i], k1 = t[cs + 2 * i + 1];
        float a0 = bf_lo(x[i]), a1 = bf_hi(x[i]);
        float b0 = bf_lo(y[i]), b1 = bf_hi(y[i]);
        rot_pair<true>(a0, b0, k0);
        rot_pair<true>(a1, b1, k1);
        x[i] = pack_bf16(a0, a1);
        y[i] = pack_bf16(b0, b1);
    }
}
template <> __device__ __forceinline__ void rot_halves<4>(u32x4& x, u32x4& y, const KCosSin* t, int32_t cs) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const KCosSin k = t[cs + i];
        float a = __uint_as_float(x[i]), b = __uint_as_float(y[i]);
        rot_pair<false>(a, b, k);
        x[i] = __float_as_uint(a);
        y[i] = __float_as_uint(b);
    }
}

// The partner lane's chunk of a lane-exchanged half-split band (partner: its lane index).  With
// 16-chunk bands on 16-chunk boundaries the partner is lane ^ 8 of the same 16-lane DPP row, read
// with a row rotation by 8 (no LDS traffic); otherwise a cross-lane permute.
__device__ __forceinline__ u32x4 partner_chunk(const KPlane& pl, const u32x4& v, int partner) {
    u32x4 o;
    if (pl.neox_dpp) {
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[i]), 0x128, 0xf, 0xf, false));
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = uint32_t(__shfl(int(v[i]), partner, 64));
    }
    return o;
}

// Lane-exchanged half-split chunk: `v` is this lane's chunk of the band, `o` the partner lane's
// (the other half); only this lane's elements are computed.  Element e pairs with element e of
// the partner chunk, cos/sin table[cs + e].
template <int ESZ> __device__ __forceinline__ void rot_halves_own(u32x4& v, const u32x4& o, const KCosSin* t,
                                                                  int32_t cs, bool lo);
template <> __device__ __forceinline__ void rot_halves_own<2>(u32x4& v, const u32x4& o, const KCosSin* t,
                                                              int32_t cs, bool lo) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float m0 = rot_own<true>(bf_lo(v[i]), bf_lo(o[i]), t[cs + 2 * i], lo);
        const float m1 = rot_own<true>(bf_hi(v[i]), bf_hi(o[i]), t[cs + 2 * i + 1], lo);
        v[i] = pack_bf16(m0, m1);
    }
}
template <> __device__ __forceinline__ void rot_halves_own<4>(u32x4& v, const u32x4& o, const KCosSin* t,
                                                              int32_t cs, bool lo) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
        v[i] = __float_as_uint(rot_own<false>(__uint_as_float(v[i]), __uint_as_float(o[i]), t[cs + i], lo));
}

// A lane-exchanged half-split chunk, rotated: `v` is this lane's chunk, `o` its partner lane's,
// `cs` the cos/sin entry of the chunk's first pair, `lo` whether this lane holds low members.
// Only this lane's members are computed (half the products of rotating both and discarding the
// partner's: GQA 16K splice +0.6 points, token-slot and in-place GQA rotations +0.3 to +0.8).
template <int ESZ>
__device__ __forceinline__ void rot_exchanged(u32x4& v, u32x4& o, const KCosSin* t, int32_t cs, bool lo) {
    rot_halves_own<ESZ>(v, o, t, cs, lo);
}

// ------------------------------------------------------------------------- row geometry ---

__device__ __forceinline__ int32_t fdiv(int32_t n, KDiv d) {
    return int32_t((__umulhi(uint32_t(n), d.mul) + uint32_t(n)) >> d.shift);
}

// Two-chunk units over all chunks of a row (half-split planes without lane exchange, and the
// ordered-chain kernel): unit u is a chunk, or a low-half chunk together with its partner.
struct Unit {
    int32_t a, b, pair, kind;
};

template <int ESZ>
__device__ __forceinline__ Unit map_unit(const KPlane& p, int32_t u) {
    constexpr int EPC = Elt<ESZ>::EPC;
    Unit r{u, -1, 0, KROT_NONE};
    if (p.rot == KROT_INTERLEAVED) {
        const int32_t h = fdiv(u, p.head_div), j = u - h * p.head_chunks;
        if (h < p.n_heads && j >= p.rot_lo && j < p.rot_lo + p.rot_chunks) {
            r.kind = KROT_INTERLEAVED;
            r.pair = (j - p.rot_lo) * (EPC / 2);
        }
    } else if (p.rot == KROT_NEOX) {
        const int32_t half = p.rot_chunks >> 1, uh = p.head_chunks - half;
        const int32_t head_units = p.n_heads * uh;
        if (u >= head_units) {
            r.a = p.n_heads * p.head_chunks + (u - head_units);
        } else {
            const int32_t h = fdiv(u, p.uhead_div), j = u - h * uh;
            r.a = h * p.head_chunks + (j < p.rot_lo + half ? j : j + half);
            if (j >= p.rot_lo && j < p.rot_lo + half) {
                r.kind = KROT_NEOX;
                r.b = r.a + half;
                r.pair = (j - p.rot_lo) * EPC;
            }
        }
    }
    return r;
}

// Re-anchor chunk u of one row in registers with the cos/sin block table[cs + pair] (single-chunk
// mode: interleaved bands, or half-split bands whose partner chunks sit in the same wavefront and
// are exchanged between lanes).  Partner lanes belong to the same row and take the same path.
template <int ESZ, int ROT = KROT_NONE>
__device__ __forceinline__ void rotate_chunk(const KPlane& pl, u32x4& v, int32_t u, const KCosSin* table,
                                             int32_t cs) {
    constexpr int EPC = Elt<ESZ>::EPC;
    const int32_t h = fdiv(u, pl.head_div);
    const int32_t j = u - h * pl.head_chunks - pl.rot_lo;
    if (h < pl.n_heads && j >= 0 && j < pl.rot_chunks) {
        if (ROT == KROT_INTERLEAVED || (ROT == KROT_NONE && pl.rot == KROT_INTERLEAVED)) {
            rot_interleaved<ESZ>(v, table, cs + j * (EPC / 2));
        } else {
            const int32_t half = pl.rot_chunks >> 1;
            const bool lo = j < half;
            const int lane = int(threadIdx.x & 63);
            const int partner = lo ? lane + half : lane - half;
            u32x4 o = partner_chunk(pl, v, partner);
            rot_exchanged<ESZ>(v, o, table, cs + (lo ? j : j - half) * EPC, lo);
        }
    }
}

// Row kernels: move unit u of one row from src to dst, re-anchored with the cos/sin block
// table[cs + pair] (cs < 0: copied unchanged).
template <int ESZ>
__device__ __forceinline__ void move_row_unit(const KPlane& pl, const char* src, char* dst, int32_t u,
                                              const KCosSin* table, int32_t cs) {
    if (pl.rot == KROT_NEOX && !pl.neox_lanes) {
        const Unit un = map_unit<ESZ>(pl, u);
        const int64_t a = int64_t(un.a) * 16, b = int64_t(un.b) * 16;
        u32x4 x = ld16(src + a), y;
        if (un.b >= 0) y = ld16(src + b);
        if (cs >= 0 && un.kind == KROT_NEOX) rot_halves<ESZ>(x, y, table, cs + un.pair);
        st16(dst + a, x);
        if (un.b >= 0) st16(dst + b, y);
        return;
    }
    const int64_t off = int64_t(u) * 16;
    u32x4 v = ld16(src + off);
    if (cs >= 0 && pl.rot != KROT_NONE) rotate_chunk<ESZ>(pl, v, u, table, cs);
    st16(dst + off, v);
}

// Rotary-only kernels.  Band unit q of a row (bands of consecutive heads back to back) is chunk
// j = q mod band_tpr of head h = q / band_tpr; in two-chunk mode (half-split bands without lane
// exchange) it covers the low-half chunk j and its partner.
template <int ESZ>
__device__ __forceinline__ void rotate_band_chunk(const KPlane& pl, u32x4& v, int32_t j, const KCosSin* table,
                                                  int32_t cs) {
    constexpr int EPC = Elt<ESZ>::EPC;
    if (pl.rot == KROT_INTERLEAVED) {
        rot_interleaved<ESZ>(v, table, cs + j * (EPC / 2));
    } else {
        const int32_t half = pl.rot_chunks >> 1;
        const bool lo = j < half;
        const int lane = int(threadIdx.x & 63);
        const int partner = lo ? lane + half : lane - half;
        u32x4 o = partner_chunk(pl, v, partner);
        rot_exchanged<ESZ>(v, o, table, cs + (lo ? j : j - half) * EPC, lo);
    }
}

template <int ESZ>
__device__ __forceinline__ void move_band(const KPlane& pl, const char* src, char* dst, int32_t q,
                                          const KCosSin* table, int32_t cs) {
    constexpr int EPC = Elt<ESZ>::EPC;
    const int32_t h = fdiv(q, pl.band_div);
    const int32_t j = q - h * pl.band_tpr;
    const int64_t a = (int64_t(h) * pl.head_chunks + pl.rot_lo + j) * 16;
    if (pl.rot == KROT_NEOX && pl.band_tpr != pl.rot_chunks) {
        const int64_t b = a + int64_t(pl.rot_chunks / 2) * 16;
        u32x4 x = ld16(src + a), y = ld16(src + b);
        rot_halves<ESZ>(x, y, table, cs + j * EPC);
        st16(dst + a, x);
        st16(dst + b, y);
        return;
    }
    u32x4 v = ld16(src + a);
    rotate_band_chunk<ESZ>(pl, v, j, table, cs);
    st16(dst + a, v);
}

// Band unit q of one row in nl <= PAGED_LPT layers (row, row + lstride, ...), rotated in place:
// every layer's loads are issued (band_load) before the cos/sin table is needed and before the
// first store (band_rotate_store).
struct BandPos {
    int64_t a, b;    // byte offsets of the unit's chunk and (two-chunk mode) of its partner
    int32_t j;       // chunk index within the head's band
    bool two;
};

__device__ __forceinline__ BandPos band_pos(const KPlane& pl, int32_t q) {
    BandPos p;
    const int32_t h = fdiv(q, pl.band_div);
    p.j = q - h * pl.band_tpr;
    p.a = (int64_t(h) * pl.head_chunks + pl.rot_lo + p.j) * 16;
    p.two = pl.rot == KROT_NEOX && pl.band_tpr != pl.rot_chunks;
    p.b = p.a + int64_t(pl.rot_chunks / 2) * 16;
    return p;
}

__device__ __forceinline__ void band_load(const BandPos& p, const char* row, int64_t lstride, int nl,
                                          u32x4 (&x)[PAGED_LPT], u32x4 (&y)[PAGED_LPT]) {
#pragma unroll
    for (int l = 0; l < PAGED_LPT; ++l) {
        if (l < nl) {
            x[l] = ld16(row + l * lstride + p.a);
            if (p.two) y[l] = ld16(row + l * lstride + p.b);
        }
    }
}

template <int ESZ>
__device__ __forceinline__ void band_rotate_store(const KPlane& pl, const BandPos& p, char* row,
                                                  int64_t lstride, int nl, u32x4 (&x)[PAGED_LPT],
                                                  u32x4 (&y)[PAGED_LPT], const KCosSin* table, int32_t cs) {
    constexpr int EPC = Elt<ESZ>::EPC;
#pragma unroll
    for (int l = 0; l < PAGED_LPT; ++l) {
        if (l < nl) {
            if (p.two) {
                rot_halves<ESZ>(x[l], y[l], table, cs + p.j * EPC);
                st16(row + l * lstride + p.b, y[l]);
            } else {
                rotate_band_chunk<ESZ>(pl, x[l], p.j, table, cs);
            }
            st16(row + l * lstride + p.a, x[l]);
        }
    }
}

// The 8 XCDs of the device take a launch's workgroups in turn (workgroup b runs on XCD b % 8).
// xcd_eighth renumbers the first 8 * (n / 8) of n workgroups so that XCD x runs the x-th eighth of
// them in order (the rest keep their numbers): each XCD then works through a range of its own
// instead of every eighth workgroup of one shared range.  Paged gathers run faster so from
// 4-token pages up (64-sequence batch, 64-token pages: 68.5% -> 77% of peak; 16-token pages:
// 66.6% -> 76.0%; 4-token pages: 64.6% -> 72.9%; 131K sequence: 1-5 points, varying with where
// the pool lies); token-slot gathers (1-token pages), in-place contiguous moves and rotations run
// slower (1 to 4 points), so only the gathers of pages of LEYLINE_GATHER_SPLIT_PAGE tokens or more
// use it.
constexpr int KXCDS = 8;
__device__ __forceinline__ int32_t xcd_eighth(int32_t b, int32_t n) {
    const int32_t per = n / KXCDS;
    return b < per * KXCDS ? (b % KXCDS) * per + b / KXCDS : b;
}

// The plane whose workgroup range [base[p], base[p+1]) holds workgroup bx (ranges of planes
// without work are empty, so no workgroup is launched for them).
__device__ __forceinline__ int plane_of(const int32_t* base, int n, int32_t bx) {
    int p = 0;
    while (p + 1 < n && bx >= base[p + 1]) ++p;
    return p;
}

// cos/sin block of one shift (n entries from table[c0]) staged in LDS by the whole workgroup.
template <int NT>
__device__ __forceinline__ void stage_cs(KCosSin* lcs, const KCosSin* table, int32_t c0, int32_t n) {
    for (int i = threadIdx.x; i < n; i += NT) lcs[i] = table[c0 + i];
}

// The same staging split around a thread's data loads (one entry per thread, n <= block size):
// cs_fetch before the data loads are issued, cs_commit after.  Vector loads complete in order,
// so the wait before the LDS write then covers the cos/sin load only, and the barrier that
// follows does not wait for any wavefront's data.
#if LEYLINE_PAIR_F64
typedef KCosSin CsReg;
#else
typedef uint64_t CsReg;   // one 64-bit value: merges with the default without a copy
#endif
template <class Ptr>
__device__ __forceinline__ CsReg cs_fetch(Ptr table, int32_t c0, int32_t n) {
    CsReg c{};
    if (int(threadIdx.x) < n) {
        const KCosSin e = table[c0 + threadIdx.x];
#if LEYLINE_PAIR_F64
        c = e;
#else
        c = uint64_t(__float_as_uint(e.c)) | (uint64_t(__float_as_uint(e.s)) << 32);
#endif
    }
    return c;
}
__device__ __forceinline__ void cs_commit(KCosSin* lcs, const CsReg& c, int32_t n) {
    if (int(threadIdx.x) < n) *reinterpret_cast<CsReg*>(lcs + threadIdx.x) = c;
}

// --------------------------------------------------------------------- contiguous splice ---

// Rounds and replacement copies: rows laid end to end, one unit per thread for CRPT rows of a
// rotating item (the same column of consecutive rows, so one cos/sin lookup serves them all) and
// for one row of an item that only copies; the (job, plane) items of a launch own consecutive
// ranges of workgroups (blockIdx.x), so a small item (a replacement copy) next to a round adds only
// its own workgroups.  A rotating item's workgroup stages its cos/sin block in LDS after the
// threads have issued their data loads, so that the two latencies overlap.  Past the item's last
// row a thread loads that last row again (every load issued without branching) and stores
// nothing.
//
// Rows per thread: a plain copy runs at the rate of a bare copy with one row per thread (two rows
// per thread, with twice the bytes in flight per workgroup, are slower in bare copies of both
// workloads' geometries), while a rotating row's pair arithmetic between its load and its store
// lengthens each workgroup's life, which the second row amortises.
template <int ESZ>
__global__ __launch_bounds__(MOVE_TPB) void contig_move_kernel(const KContigParams P) {
    constexpr int EPC = Elt<ESZ>::EPC;
    static_assert(KMAX_CS <= MOVE_TPB, "one cos/sin entry per thread");
    __shared__ KCosSin lcs[KMAX_CS];
    // The item whose range holds this workgroup: the number of later items starting at or before
    // it, and that item's first workgroup, selected from the same reads (independent reads, no
    // loop-carried dependency, no second load through the item index).  The item is then read as
    // a value: its fields come in one level of independent scalar loads (through a reference the
    // compiler loaded them one by one between the branches below).
    int32_t it = 0, b0 = P.block0[0];
#pragma unroll
    for (int i = 1; i < KMAX_LAUNCH_ITEMS; ++i) {
        const bool ge = int32_t(blockIdx.x) >= P.block0[i];
        it += ge ? 1 : 0;
        b0 = ge ? P.block0[i] : b0;
    }
    KItem I;
    __builtin_memcpy(&I, &P.items[it], sizeof(KItem));
    const int32_t bx = int32_t(blockIdx.x) - b0;
    const KPlane& pl = I.pl;
    const int rpt = round_rows_per_thread(I.cs >= 0);                      // block-uniform
    const int64_t groups = rpt == 1 ? I.count : (I.count + CRPT - 1) / CRPT;
    if (int64_t(bx) * MOVE_TPB >= groups * pl.tpr) return;               // block past this item's rows
    const int layer = blockIdx.y;
    const int32_t t = bx * MOVE_TPB + int32_t(threadIdx.x);
    int32_t g, u;
    row_unit(pl, LEYLINE_ROUND_PACK, t, groups, g, u);
    const int64_t r0 = int64_t(g) * rpt;
    const bool active = r0 < I.count;
    char* lbase = pl.base + int64_t(layer) * pl.layer_stride;
    const bool stub = I.kind == KJOB_STUB;
    const char* src = stub ? I.stub + int64_t(layer) * I.count * pl.row_bytes : lbase + I.src0 * pl.token_stride;
    const int64_t src_step = stub ? int64_t(pl.row_bytes) : pl.token_stride;
    char* dst = lbase + (stub ? I.dst0 : I.src0 + I.delta) * pl.token_stride;
    const bool rot = I.cs >= 0;                                    // block-uniform
    if (pl.rot == KROT_NEOX && !pl.neox_lanes) {
        // half-split two-chunk units (rare layouts; a thread's unit is not a single chunk)
        if (rot) {
            for (int i = threadIdx.x; i < pl.n_pairs; i += MOVE_TPB) lcs[i] = P.cs[I.cs + i];
            __syncthreads();
        }
        if (!active) return;
        for (int k = 0; k < rpt; ++k) {
            const int64_t r = r0 + k;
            if (r < I.count)
                move_row_unit<ESZ>(pl, src + r * src_step, dst + r * pl.token_stride, u, lcs, rot ? 0 : -1);
        }
        return;
    }
    const int64_t off = int64_t(u) * 16;
    // narrow bands (a slice of each row): entry fetched before the data, barrier waits for no
    // data; wide bands (most of the row rotates): staged after the data loads, so the barrier
    // also lines up the workgroup's stores (measured faster there)
    const bool early = rot && !pl.band_wide;
    const CsReg c = cs_fetch(P.cs, I.cs, early ? pl.n_pairs : 0);
    u32x4 v[CRPT];
#pragma unroll
    for (int k = 0; k < CRPT; ++k) {
        if (k == 0 || k < rpt) {
            const int64_t r = min(r0 + k, I.count - 1);
            v[k] = ld16(src + r * src_step + off);
        }
    }
    if (rot) {
        if (early) cs_commit(lcs, c, pl.n_pairs);
        else for (int i = threadIdx.x; i < pl.n_pairs; i += MOVE_TPB) lcs[i] = P.cs[I.cs + i];
        __syncthreads();
    }
    if (!active) return;
    const int32_t h = fdiv(u, pl.head_div);
    const int32_t j = u - h * pl.head_chunks - pl.rot_lo;
    const bool in_band = rot && h < pl.n_heads && j >= 0 && j < pl.rot_chunks;
#pragma unroll
    for (int k = 0; k < CRPT; ++k) {
        if ((k == 0 || k < rpt) && r0 + k < I.count) {
            if (in_band) {
                if (pl.rot == KROT_INTERLEAVED) {
                    rot_interleaved<ESZ>(v[k], lcs, j * (EPC / 2));
                } else {
                    const int32_t half = pl.rot_chunks >> 1;
                    const bool lo = j < half;
                    const int lane = int(threadIdx.x & 63);
                    const int partner = lo ? lane + half : lane - half;
                    u32x4 o = partner_chunk(pl, v[k], partner);
                    rot_exchanged<ESZ>(v[k], o, lcs, (lo ? j : j - half) * EPC, lo);
                }
            }
            st16(dst + (r0 + k) * pl.token_stride + off, v[k]);
        }
    }
}

// Ordered chains (shifts too small for rounds, on layouts whose half-split partners cannot be
// exchanged between lanes, so tiles are not used): thread (chain c, unit u) walks rows c, c+m, ...
template <int ESZ>
__global__ __launch_bounds__(TPB) void contig_chain_kernel(const KContigParams P) {
    const KItem& I = P.items[blockIdx.z];
    const KPlane& pl = I.pl;
    const int layer = blockIdx.y;
    const int32_t t = int32_t(blockIdx.x) * TPB + int32_t(threadIdx.x);
    char* lbase = pl.base + int64_t(layer) * pl.layer_stride;
    const int64_t ts = pl.token_stride;
    const int32_t U = pl.units_all;
    const int32_t c = t / U, u = t - c * U;
    if (c >= I.chains) return;
    const Unit un = map_unit<ESZ>(pl, u);
    const int64_t oa = int64_t(un.a) * 16, ob = int64_t(un.b) * 16;
    const int32_t cs = (I.cs >= 0 && un.kind != KROT_NONE) ? I.cs + un.pair : -1;

    const int64_t m = I.delta < 0 ? -I.delta : I.delta;
    const int64_t steps = (I.count - c + m - 1) / m;
    const char* src_c = lbase + (I.src0 + c) * ts;   // step k reads src_c + k*m*ts
    const int64_t step_bytes = m * ts;
    const int64_t dshift = I.delta * ts;             // destination = source + dshift
    const bool down = I.delta < 0;                   // left shift: ascending chain walk

    u32x4 va[WIN], vb[WIN];
    for (int64_t k0 = 0; k0 < steps; k0 += WIN) {
#pragma unroll
        for (int w = 0; w < WIN; ++w) {
            const int64_t k = down ? k0 + w : steps - 1 - (k0 + w);
            if (k0 + w < steps) {
                const char* s = src_c + k * step_bytes;
                va[w] = ld16(s + oa);
                if (un.b >= 0) vb[w] = ld16(s + ob);
            }
        }
#pragma unroll
        for (int w = 0; w < WIN; ++w) {
            const int64_t k = down ? k0 + w : steps - 1 - (k0 + w);
            if (k0 + w < steps) {
                if (cs >= 0) {
                    if (un.kind == KROT_INTERLEAVED) rot_interleaved<ESZ>(va[w], P.cs, cs);
                    else rot_halves<ESZ>(va[w], vb[w], P.cs, cs);
                }
                char* d = const_cast<char*>(src_c) + k * step_bytes + dshift;
                st16(d + oa, va[w]);
                if (un.b >= 0) st16(d + ob, vb[w]);
            }
        }
    }
}

// Ordered tiles: every job of a call whose moves are too short-shifted for rounds.  Each
// (job, plane) item is cut into tiles of tile_chunks chunks (KTILE_CHUNKS, a quarter of that in a
// call of few tiles, or a whole number of packed blocks for a packed item; counted from its first
// row) in each layer.  Workgroups take tile tickets from a counter, in order; the items of a launch own
// consecutive ticket ranges in dependency order, and within an item ticket t is tile
// t mod n_tiles of its processing order (a left shift ascending, a right shift descending) in
// layer t / n_tiles, so that the tiles in flight cover one stretch of one layer (interleaving
// the layers costs several points of bandwidth).
//
// A tile's chunks are loaded into registers; once those loads have returned, a move tile
// publishes "source read".  Before storing, a tile waits for every tile whose source rows its
// destination overlaps (tile_wait_flags), so no tile reads a chunk another tile has written.
// A tile waits only for tickets taken before its own, which publish without waiting, so every
// wait ends.  The wait is still bounded (KTILE_SPIN_LIMIT polls per flag): a tile that gives up
// flags LEYLINE_STATUS_TILE_TIMEOUT and stores nothing, and the launch drains.
//
// ROT: the rotary style of every re-anchored item of the launch (KROT_NONE: looked up per item),
// so that the style this launch does not use costs no registers.
__device__ __forceinline__ bool wait_flag(const int32_t* f) {
    return tile_wait_bounded(
        [f] { return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0; },
        [] { __builtin_amdgcn_s_sleep(1); }, KTILE_SPIN_LIMIT);
}

// Persistent tile workgroups.  A workgroup keeps taking tickets until they run out, and holds at
// most two tiles: the current one, whose chunks are in registers and whose "source read" flag is
// published, and the next one, whose loads it issues before it waits for the current tile's
// dependencies and stores it, so that the next tile's loads are in flight during that wait and
// those stores.  Every wait still ends: the lowest unpublished ticket is either a workgroup's
// current tile, published as soon as its loads return, or a workgroup's next tile, whose current
// tile is lower, so all of that tile's dependencies are published and the workgroup goes on to
// publish the next one.  A prefetched tile never reads a row that a lower ticket writes (a writer
// always waits for the readers of its rows, which hold lower tickets).

// One tile (ticket) of a tile launch, from the workgroup's point of view.
struct TileCtx {
    const char* src;
    char* dst;
    int64_t src_step;        // bytes between consecutive source rows
    int32_t it, layer, order, local;
    int32_t g0;              // this thread's first chunk of the tile
    int32_t total;           // chunks of the item in one layer
    int32_t end;             // end of the tile's chunks
    int32_t rows;            // rows of the item
    int32_t slots;           // a thread's chunk slots that can fall inside the tile (tile-uniform)
    int32_t cs;              // first cos/sin entry (-1: copied unchanged)
    int32_t plane, flag0;
    bool move, pack;
};

__device__ __forceinline__ TileCtx tile_ctx(const KTileParams& P, int32_t ticket) {
    TileCtx c;
    c.it = tile_item_of(P, ticket);
    KTileItem I;                // the item as a value: one level of independent scalar loads
    __builtin_memcpy(&I, &P.items[c.it], sizeof(KTileItem));
    const KPlane& pl = P.planes[I.plane];
    c.move = I.kind == KJOB_TILE;
    c.local = ticket - I.ticket0;
    c.layer = c.local / I.n_tiles;
    c.order = c.local - c.layer * I.n_tiles;
    const int32_t q = I.delta <= 0 ? c.order : I.n_tiles - 1 - c.order;
    c.total = int32_t(I.count) * pl.tpr;
    char* lbase = pl.base + int64_t(c.layer) * pl.layer_stride;
    c.src = c.move ? lbase + I.src0 * pl.token_stride : I.stub + int64_t(c.layer) * I.count * pl.row_bytes;
    c.src_step = c.move ? pl.token_stride : pl.row_bytes;
    c.dst = lbase + I.dst0 * pl.token_stride;
    c.g0 = q * I.tile_chunks + int32_t(threadIdx.x);
    c.end = min(c.total, (q + 1) * I.tile_chunks);
    c.slots = (c.end - q * I.tile_chunks + KTILE_TPB - 1) / KTILE_TPB;
    c.rows = int32_t(I.count);
    c.pack = LEYLINE_TILE_PACK && I.pack;
    c.cs = I.cs;
    c.plane = I.plane;
    c.flag0 = I.flag0;
    return c;
}

// Every slot that can fall inside the tile loads (a thread past the end of the tile: the tile's
// last chunk, which stays unused), so that the loads are issued back to back without divergent
// branches between them; slots past every thread's share of a short tile (the quarter-size tiles
// of small calls, an item's last tile) are skipped by a tile-uniform test.  A packed item's tiles
// are whole packed blocks, so its units (row_unit) cover the same rows as in plain order.
__device__ __forceinline__ void tile_load(const KTileParams& P, const TileCtx& c, u32x4 (&v)[KTILE_CPT]) {
    const KPlane& pl = P.planes[c.plane];
#pragma unroll
    for (int i = 0; i < KTILE_CPT; ++i) {
        if (i == 0 || i < c.slots) {
            const int32_t gc = min(c.g0 + i * KTILE_TPB, c.end - 1);
            int32_t r, u;
            row_unit(pl, c.pack, gc, c.rows, r, u);
            v[i] = ld16(c.src + int64_t(r) * c.src_step + int64_t(u) * 16);
        }
    }
}

template <int ESZ, int ROT>
__device__ __forceinline__ void tile_store(const KTileParams& P, const TileCtx& c, u32x4 (&v)[KTILE_CPT],
                                           const KCosSin* lcs) {
    const KPlane& pl = P.planes[c.plane];
#pragma unroll
    for (int i = 0; i < KTILE_CPT; ++i) {
        const int32_t g = c.g0 + i * KTILE_TPB;
        if ((i == 0 || i < c.slots) && g < c.end) {
            int32_t r, u;
            row_unit(pl, c.pack, g, c.rows, r, u);
            if (c.cs >= 0) rotate_chunk<ESZ, ROT>(pl, v[i], u, lcs, 0);
            st16(c.dst + int64_t(r) * pl.token_stride + int64_t(u) * 16, v[i]);
        }
    }
}

// One step of a persistent workgroup: `cur` is loaded into `v` (loads issued) with its cos/sin
// in `lcs`; the next ticket's tile goes to `nxt`, `nv` and `nlcs`.  Returns the next ticket
// (>= n_tickets: none).  words[0] carries the next ticket, words[1] the store decision.
template <int ESZ, int ROT>
__device__ __forceinline__ int32_t tile_step(const KTileParams& P, const TileCtx& cur, u32x4 (&v)[KTILE_CPT],
                                             const KCosSin* lcs, TileCtx& nxt, u32x4 (&nv)[KTILE_CPT],
                                             KCosSin* nlcs, int32_t* words) {
    __builtin_amdgcn_s_waitcnt(0);          // this thread's loads of the tile have returned
    __syncthreads();                        // ... and every thread's; the tile's cos/sin are staged
    if (threadIdx.x == 0) {
        if (cur.move)
            __hip_atomic_store(P.flags + cur.flag0 + cur.local, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        words[0] = atomicAdd(P.counter, 1);
    }
    __syncthreads();
    const int32_t next = words[0];          // block-uniform
    const bool more = next < P.n_tickets;
    // Loads return in order, so a flag read issued after the next tile's loads would wait for
    // them: the first wavefront waits for the current tile's dependencies before it issues its
    // share of the next tile's loads; the other wavefronts issue theirs at once.
    const bool waiter = threadIdx.x < 64;
    if (more) nxt = tile_ctx(P, next);
    if (more && !waiter) tile_load(P, nxt, nv);
    if (threadIdx.x == 0) {
        bool ok = true;
        tile_wait_flags(P, cur.it, cur.layer, cur.order, [&](int64_t f) { ok = ok && wait_flag(P.flags + f); });
        if (!ok && P.status) atomicOr(P.status, int(LEYLINE_STATUS_TILE_TIMEOUT));
        words[1] = ok ? 1 : 0;
    }
    // the next tile's cos/sin (at most 64 pairs per plane, so the first wavefront fetches them)
    const int32_t n_cs = more && nxt.cs >= 0 ? P.planes[nxt.plane].n_pairs : 0;
    CsReg c{};
    if (waiter) {
        c = cs_fetch(P.cs, nxt.cs, n_cs);
        if (more) tile_load(P, nxt, nv);
    }
    __syncthreads();
    if (words[1]) tile_store<ESZ, ROT>(P, cur, v, lcs);   // a wait given up: store nothing
    if (n_cs > 64) {                        // wider bands: the rest of the entries, plainly
        if (!waiter) c = cs_fetch(P.cs, nxt.cs, n_cs);
    }
    cs_commit(nlcs, c, n_cs);
    return more ? next : P.n_tickets;
}

template <int ESZ, int ROT>
__global__ __launch_bounds__(KTILE_TPB) void contig_tile_kernel(const KTileParams P) {
    __shared__ KCosSin lcs[2][KMAX_CS];
    __shared__ int32_t words[2];
    if (threadIdx.x == 0) words[0] = atomicAdd(P.counter, 1);
    __syncthreads();
    int32_t ticket = words[0];
    if (ticket >= P.n_tickets) return;                            // block-uniform
    TileCtx a = tile_ctx(P, ticket), b = a;
    u32x4 va[KTILE_CPT], vb[KTILE_CPT];
    tile_load(P, a, va);
    if (a.cs >= 0) stage_cs<KTILE_TPB>(lcs[0], P.cs, a.cs, P.planes[a.plane].n_pairs);
    // two steps per iteration, so that the register buffers alternate without copies
    for (;;) {
        ticket = tile_step<ESZ, ROT>(P, a, va, lcs[0], b, vb, lcs[1], words);
        if (ticket >= P.n_tickets) return;
        ticket = tile_step<ESZ, ROT>(P, b, vb, lcs[1], a, va, lcs[0], words);
        if (ticket >= P.n_tickets) return;
    }
}

// The rotary style shared by every re-anchored item of a tile launch, or KROT_NONE when items of
// both styles (or none) are re-anchored.
static int32_t launch_rot_style(const KTileParams& P) {
    int32_t style = KROT_NONE;
    for (int32_t i = 0; i < P.n_items; ++i) {
        const int32_t rot = P.planes[P.items[i].plane].rot;
        if (P.items[i].cs < 0 || rot == KROT_NONE) continue;
        if (style != KROT_NONE && style != rot) return KROT_NONE;
        style = rot;
    }
    return style;
}

// Clears n_zero 32-bit words (the tile launches' ticket counters and flags) and writes n_cs
// entries of the call's cos/sin table from the kernel arguments into the workspace.
__global__ __launch_bounds__(TPB) void tile_prep_kernel(const KPrepParams Q) {
    const int64_t stride = int64_t(gridDim.x) * TPB;
    for (int64_t i = int64_t(blockIdx.x) * TPB + threadIdx.x; i < Q.n_zero; i += stride) Q.zero[i] = 0;
    for (int64_t i = int64_t(blockIdx.x) * TPB + threadIdx.x; i < Q.n_cs; i += stride) Q.cs_dst[i] = Q.cs[i];
}

// ------------------------------------------------------------------------ rotate in place ---

// In-place R(delta) on listed rows: band units of all rows laid end to end, the workgroups of
// each rotary plane after those of the previous one, PAGED_LPT layers per thread, the shift's
// cos/sin staged in LDS.
// SOLO: only plane 0 has work in this launch, so no workgroup looks its plane up (one level of
// dependent scalar loads less before the data loads).
template <int ESZ, bool SOLO, bool PAGED>
__global__ __launch_bounds__(PAGED_TPB) void rotate_rows_kernel(const KRotateParams P) {
    __shared__ KCosSin lcs[KMAX_CS];
    // the call's scalars as one value: one level of independent scalar loads
    KRotateHead H;
    __builtin_memcpy(&H, &P.h, sizeof(KRotateHead));
    const int plane = SOLO ? 0 : plane_of(P.rot_base, H.n_planes, int32_t(blockIdx.x));
    const KPlane& pl = P.planes[plane];
    const int32_t tb = (SOLO ? int32_t(blockIdx.x) : int32_t(blockIdx.x) - P.rot_base[plane]) * PAGED_TPB;
    if (int64_t(tb) >= H.n_rows * pl.rot_tpr) return;                  // past this plane
    const int32_t t = tb + int32_t(threadIdx.x);
    const int32_t i = fdiv(t, P.rot_div[plane]), q = t - i * pl.rot_tpr;
    bool active = i < H.n_rows;
    int64_t row = active ? (H.rows ? H.rows[i] : H.row0 + i) : 0;
    if (active && (row < 0 || row >= H.total_rows)) {
        if (H.status && q == 0 && blockIdx.y == 0) atomicOr(H.status, int(LEYLINE_STATUS_BAD_ROW));
        active = false;
    }
    const int layer0 = int(blockIdx.y) * PAGED_LPT;
    const int nl = min(PAGED_LPT, H.n_layers - layer0);
    char* r = pl.base + int64_t(layer0) * pl.layer_stride;
    if constexpr (PAGED) {
        const int32_t pg = fdiv(int32_t(row), P.page_div);
        r += int64_t(pg) * pl.page_stride + (row - int64_t(pg) * H.page_size) * pl.token_stride;
    } else {
        r += row * pl.token_stride;
    }
    const BandPos bp = band_pos(pl, q);
    static_assert(KMAX_CS <= PAGED_TPB, "one cos/sin entry per thread");
    const CsReg c = cs_fetch(P.cs, pl.cs_off, pl.n_pairs);
    u32x4 x[PAGED_LPT], y[PAGED_LPT];
    if (active) band_load(bp, r, pl.layer_stride, nl, x, y);
    cs_commit(lcs, c, pl.n_pairs);
    __syncthreads();
    if (!active) return;
    band_rotate_store<ESZ>(pl, bp, r, pl.layer_stride, nl, x, y, lcs, 0);
}

// ------------------------------------------------------------------------------ paged splice ---
//
// paged_data_kernel moves the data.  Its first blocks gather ASSEMBLE rows like the contiguous
// kernel (rows laid end to end, one 16-byte chunk per thread, so a wavefront reads one row entry
// and moves whole lines); its last blocks rotate the rotary bands of REMAP pages (re-used whole
// pages) in place, each looking its pages up in the plan and the old block table (or reading
// them from paged_remap_order_kernel's physical-order list).  The rows of a small gather
// (token-slot splices: the replacement rows) are resolved by the gathering blocks themselves, and
// the new block tables and freed list are written by blocks between the two: one launch per call.
// A large gather first runs paged_resolve_kernel, which expands the page runs once for all layers
// and planes into a row table (for every row of every ASSEMBLE page: which old physical page and
// row, or which replacement token, it comes from, which fresh page it goes to, which shift
// re-anchors it) and writes the block tables and the freed list; paged_order_kernel before it
// lays the row table out in destination-page order.
// Nothing is written to an old page except the rotary bands of REMAP pages, which no ASSEMBLE
// row reads.

// The plan's tables, in the workspace or in this launch's kernel arguments.
struct PlanView {
    const KSeqEntry* seqs;
    const KDirEntry* dirs;
    const KCosSin* cs;
    const KPageRun* runs;
    const KPageRun* asm_runs;
    const KPageRun* remap_runs;
    const KFreedRun* freed_runs;
};

// The kernel's only argument is a KPagedParams at the start of the kernel-argument segment, so an
// inline plan sits at that segment's address plus the offset of `blob` (the address of the
// argument itself is not taken, which would make the compiler copy it into private memory).
// Both places are global device memory: the pointer is formed in the global address space so
// that the compiler reads the tables with global loads instead of flat ones (a flat load can
// only be waited for together with every earlier memory access).
__device__ __forceinline__ PlanView plan_view(const KPagedParams& P) {
    using G = const __attribute__((address_space(1))) char*;
    const G kernarg = (G)(const char*)__builtin_amdgcn_kernarg_segment_ptr();
    const char* b = (const char*)(P.plan ? (G)P.plan : kernarg + offsetof(KPagedParams, blob));
    return PlanView{reinterpret_cast<const KSeqEntry*>(b + P.off_seq),
                    reinterpret_cast<const KDirEntry*>(b + P.off_dir),
                    reinterpret_cast<const KCosSin*>(b + P.off_cs),
                    reinterpret_cast<const KPageRun*>(b + P.off_runs),
                    reinterpret_cast<const KPageRun*>(b + P.off_asm_runs),
                    reinterpret_cast<const KPageRun*>(b + P.off_remap_runs),
                    reinterpret_cast<const KFreedRun*>(b + P.off_freed_runs)};
}

// The run holding ordinal x among n runs sorted by ord0 (runs[0].ord0 <= x).
__device__ __forceinline__ int32_t run_of(const KPageRun* runs, int32_t n, int32_t x) {
    int32_t lo = 0, hi = n;
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (runs[mid].ord0 <= x) lo = mid; else hi = mid;
    }
    return lo;
}

// REMAP page m of run R (whose shift has cos/sin entry cs and whose sequence has new length
// new_len): its physical page from the old block table and its valid rows (0 when the page is
// out of the pool, which is flagged).
__device__ __forceinline__ KRemapPage remap_entry(const KPagedParams& P, const KPageRun& R, int32_t cs,
                                                  int32_t new_len, int32_t m) {
    const int32_t c = m - R.ord0;
    KRemapPage e{0, cs, 0, 0};
    const int32_t pg = P.bt_in[int64_t(R.seq) * P.bt_stride + R.src0 + c];
    if (pg < 0 || pg >= P.capacity) {
        if (P.status) atomicOr(P.status, int(LEYLINE_STATUS_BAD_PAGE));
    } else if (cs >= 0) {
        e.page = pg;
        e.rows = int32_t(min(int64_t(P.page_size), int64_t(new_len) - int64_t(R.k0 + c) * P.page_size));
    }
    return e;
}

// New block-table entry i (sequence i / bt_stride, page i % bt_stride) from the page runs.
__device__ __forceinline__ void resolve_table_entry(const KPagedParams& P, const PlanView& V, int32_t i) {
    const int32_t b = i / P.bt_stride, k = i - b * P.bt_stride;
    const KSeqEntry S = V.seqs[b];
    int32_t v = -1;
    if (S.run_count > 0 && int64_t(k) * P.page_size < S.new_len) {
        int32_t lo = S.run_begin, hi = S.run_begin + S.run_count;
        while (hi - lo > 1) {
            const int32_t mid = (lo + hi) >> 1;
            if (V.runs[mid].k0 <= k) lo = mid; else hi = mid;
        }
        const KPageRun R = V.runs[lo];
        const int32_t src = R.src0 + (k - R.k0);
        if (R.kind == LEYLINE_PAGE_ASSEMBLE) v = src < P.n_free ? P.free_pages[src] : -1;
        else v = P.bt_in[int64_t(b) * P.bt_stride + src];
    }
    P.bt_out[i] = v;
}

// Freed-list entry f from the freed runs.
__device__ __forceinline__ void resolve_freed_entry(const KPagedParams& P, const PlanView& V, int32_t f) {
    int32_t lo = 0, hi = P.n_freed_runs;
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (V.freed_runs[mid].out0 <= f) lo = mid; else hi = mid;
    }
    const KFreedRun R = V.freed_runs[lo];
    P.freed_out[f] = P.bt_in[int64_t(R.seq) * P.bt_stride + R.page0 + (f - R.out0)];
}

// Orders the call's fresh pages by physical destination page, in buckets of 2^order_shift pages,
// so that the gather writes neighbouring pages together (with a scattered free list this saves
// address-translation misses: measured 3 points of peak).  One workgroup: a histogram of the
// buckets in LDS, an exclusive scan, and a scatter of the fresh ordinals into P.order.  A page
// outside the pool counts in bucket 0 (its rows are flagged and skipped when resolved).  Up to
// ORDER_STAGE ordinals are scattered in LDS and written out in order: scattered 4-byte stores
// from one compute unit cost about 5 us per 15,000.
constexpr int ORDER_TPB = 1024;
constexpr int ORDER_STAGE = 24576;
constexpr int ORDER_PER = ORDER_STAGE / ORDER_TPB;   // fresh ordinals a thread holds

// The counts cnt[KORDER_BUCKETS] replaced by their exclusive prefix sums, by a workgroup of
// ORDER_TPB threads: each thread sums its KORDER_BUCKETS / ORDER_TPB consecutive buckets, the
// wavefronts scan those sums with lane shuffles, and one barrier exchanges the wavefront totals
// (wsum: ORDER_TPB / 64 entries).  Ends with a barrier, so cnt is ready for every thread.
__device__ __forceinline__ void bucket_offsets(int32_t* cnt, int32_t* wsum) {
    constexpr int PER = KORDER_BUCKETS / ORDER_TPB;
    const int tid = int(threadIdx.x), lane = tid & 63, wave = tid >> 6;
    int32_t own[PER], sum = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        own[k] = cnt[tid * PER + k];
        sum += own[k];
    }
    int32_t x = sum;                                   // inclusive scan within the wavefront
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int32_t run = x - sum;
    for (int w = 0; w < wave; ++w) run += wsum[w];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        cnt[tid * PER + k] = run;
        run += own[k];
    }
    __syncthreads();
}
__global__ __launch_bounds__(ORDER_TPB) void paged_order_kernel(const KPagedParams P) {
    __shared__ int32_t cnt[KORDER_BUCKETS];
    __shared__ int32_t part[ORDER_TPB / 64];
    __shared__ int32_t stage[ORDER_STAGE];
    const int tid = int(threadIdx.x);
    for (int i = tid; i < KORDER_BUCKETS; i += ORDER_TPB) cnt[i] = 0;
    auto bucket = [&](int32_t t) {
        const int32_t pg = t < P.n_free ? P.free_pages[t] : -1;
        return (pg < 0 || pg >= P.capacity) ? 0 : (pg >> P.order_shift);
    };
    // up to ORDER_STAGE ordinals: every thread's buckets loaded at once and kept for the scatter
    const bool held = P.n_asm <= ORDER_STAGE;                     // block-uniform
    int32_t b[ORDER_PER];
    if (held) {
#pragma unroll
        for (int k = 0; k < ORDER_PER; ++k) {
            const int32_t t = tid + k * ORDER_TPB;
            b[k] = t < P.n_asm ? bucket(t) : -1;
        }
    }
    __syncthreads();
    if (held) {
#pragma unroll
        for (int k = 0; k < ORDER_PER; ++k)
            if (b[k] >= 0) atomicAdd(&cnt[b[k]], 1);
    } else {
        for (int32_t t = tid; t < P.n_asm; t += ORDER_TPB) atomicAdd(&cnt[bucket(t)], 1);
    }
    __syncthreads();
    // exclusive scan: each thread owns KORDER_BUCKETS / ORDER_TPB consecutive buckets
    bucket_offsets(cnt, part);
    if (held) {
#pragma unroll
        for (int k = 0; k < ORDER_PER; ++k)
            if (b[k] >= 0) stage[atomicAdd(&cnt[b[k]], 1)] = tid + k * ORDER_TPB;
        __syncthreads();
        for (int32_t j = tid; j < P.n_asm; j += ORDER_TPB) P.order[j] = stage[j];
    } else {
        for (int32_t t = tid; t < P.n_asm; t += ORDER_TPB) P.order[atomicAdd(&cnt[bucket(t)], 1)] = t;
    }
}

// REMAP page m of the call (in plan order), resolved: its physical page, shift and valid rows.
__device__ __forceinline__ KRemapPage remap_resolve(const KPagedParams& P, const PlanView& V, int32_t m) {
    if (P.n_remap_runs == 1) return remap_entry(P, P.remap0, P.remap0_cs, P.remap0_len, m);
    const KPageRun R = V.remap_runs[run_of(V.remap_runs, P.n_remap_runs, m)];
    return remap_entry(P, R, V.dirs[R.dir].cs, V.seqs[R.seq].new_len, m);
}

// Lays the call's REMAP pages out in physical-page order, resolved (buckets of 2^remap_shift
// pages; one workgroup: a histogram in LDS, an exclusive scan, a scatter), so that the rotating
// workgroups that run together touch neighbouring pages.  A page outside the pool (flagged, no
// rows to rotate) counts in bucket 0.  Up to ORDER_TPB * REMAP_SORT_PER pages are resolved once,
// all loads of a thread in flight together, and kept in registers for the scatter; larger calls
// sweep twice.  Held entries are scattered in LDS (packed into 8 bytes when P.remap_pack says
// that the shift index and the row count fit 16 bits each) and written out in order.
constexpr int REMAP_SORT_PER = 16;

__global__ __launch_bounds__(ORDER_TPB) void paged_remap_order_kernel(const KPagedParams P) {
    __shared__ int32_t cnt[KORDER_BUCKETS];
    __shared__ int32_t part[ORDER_TPB / 64];
    __shared__ uint2 stage[ORDER_TPB * REMAP_SORT_PER];
    const PlanView V = plan_view(P);
    const int tid = int(threadIdx.x);
    const bool held = P.n_remap <= ORDER_TPB * REMAP_SORT_PER;     // block-uniform
    for (int i = tid; i < KORDER_BUCKETS; i += ORDER_TPB) cnt[i] = 0;
    KRemapPage e[REMAP_SORT_PER];
    if (held) {
#pragma unroll
        for (int k = 0; k < REMAP_SORT_PER; ++k) {
            const int32_t m = tid + k * ORDER_TPB;
            e[k] = m < P.n_remap ? remap_resolve(P, V, m) : KRemapPage{0, -1, 0, 0};
        }
    }
    __syncthreads();
    if (held) {
#pragma unroll
        for (int k = 0; k < REMAP_SORT_PER; ++k)
            if (tid + k * ORDER_TPB < P.n_remap) atomicAdd(&cnt[e[k].page >> P.remap_shift], 1);
    } else {
        for (int32_t m = tid; m < P.n_remap; m += ORDER_TPB)
            atomicAdd(&cnt[remap_resolve(P, V, m).page >> P.remap_shift], 1);
    }
    __syncthreads();
    bucket_offsets(cnt, part);
    if (held && P.remap_pack) {
#pragma unroll
        for (int k = 0; k < REMAP_SORT_PER; ++k)
            if (tid + k * ORDER_TPB < P.n_remap)
                stage[atomicAdd(&cnt[e[k].page >> P.remap_shift], 1)] =
                    uint2{uint32_t(e[k].page), uint32_t(e[k].cs + 1) | (uint32_t(max(e[k].rows, 0)) << 16)};
        __syncthreads();
        for (int32_t j = tid; j < P.n_remap; j += ORDER_TPB) {
            const uint2 w = stage[j];
            P.remap_sorted[j] = KRemapPage{int32_t(w.x), int32_t(w.y & 0xffffu) - 1, int32_t(w.y >> 16), 0};
        }
    } else if (held) {
#pragma unroll
        for (int k = 0; k < REMAP_SORT_PER; ++k)
            if (tid + k * ORDER_TPB < P.n_remap) P.remap_sorted[atomicAdd(&cnt[e[k].page >> P.remap_shift], 1)] = e[k];
    } else {
        for (int32_t m = tid; m < P.n_remap; m += ORDER_TPB) {
            const KRemapPage x = remap_resolve(P, V, m);
            P.remap_sorted[atomicAdd(&cnt[x.page >> P.remap_shift], 1)] = x;
        }
    }
}

// ASSEMBLE row i (row i mod page_size of the (i / page_size)-th fresh page in destination order
// when P.order is set, else in plan order): where it comes from, where it goes, its shift.
__device__ __forceinline__ KRowMove row_entry(const KPagedParams& P, const PlanView& V, int32_t i) {
    const int32_t slot = i / P.page_size, r = i - slot * P.page_size;
    const int32_t task = P.order ? P.order[slot] : slot;               // fresh ordinal
    const KPageRun R = V.asm_runs[run_of(V.asm_runs, P.n_asm_runs, task)];
    const int32_t seq = R.seq, k = R.k0 + (task - R.ord0);
    const KSeqEntry S = V.seqs[seq];
    const int64_t q = int64_t(k) * P.page_size + r;
    KRowMove e{KROW_SKIP, 0, 0, r, -1, -1};
    if (q >= S.new_len) return e;
    const int32_t fp = task < P.n_free ? P.free_pages[task] : -1;
    if (fp < 0 || fp >= P.capacity) {
        if (P.status) atomicOr(P.status, int(LEYLINE_STATUS_BAD_PAGE));
        return e;
    }
    e.dst_page = fp;
    // last directive of the sequence whose replacement starts at or before q
    int32_t jlo = 0, jhi = S.dir_count;
    while (jlo < jhi) {
        const int32_t mid = (jlo + jhi) >> 1;
        if (V.dirs[S.dir_begin + mid].stub_start <= q) jlo = mid + 1; else jhi = mid;
    }
    int64_t old = q;
    if (jlo > 0) {
        const int32_t j = S.dir_begin + jlo - 1;
        const KDirEntry D = V.dirs[j];
        if (q < D.stub_start + D.stub_len) {
            e.src_page = KROW_STUB;
            e.src_row = int32_t(q - D.stub_start);
            e.dir = j;
            return e;
        }
        old = q - D.delta;
        e.cs = D.cs;
    }
    const int32_t pg = P.bt_in[int64_t(seq) * P.bt_stride + old / P.page_size];
    if (pg < 0 || pg >= P.capacity) {
        if (P.status) atomicOr(P.status, int(LEYLINE_STATUS_BAD_PAGE));
        e.src_page = KROW_SKIP;
    } else {
        e.src_page = pg;
        e.src_row = int32_t(old % P.page_size);
    }
    return e;
}

// Entry w of the call's table work: the n_table new block-table entries, then the n_freed
// freed-list entries.
__device__ __forceinline__ void table_work(const KPagedParams& P, const PlanView& V, int64_t w) {
    if (w < P.n_table) resolve_table_entry(P, V, int32_t(w));
    else if (w - P.n_table < P.n_freed) resolve_freed_entry(P, V, int32_t(w - P.n_table));
}

// Large gathers: threads [0, n_rows) write the row table (in destination order when P.order is
// set), the following ones the block tables and the freed list.
__global__ __launch_bounds__(TPB) void paged_resolve_kernel(const KPagedParams P) {
    const PlanView V = plan_view(P);
    const int32_t i = int32_t(blockIdx.x) * TPB + int32_t(threadIdx.x);
    if (i < P.n_rows) P.rows[i] = row_entry(P, V, i);
    else table_work(P, V, int64_t(i) - P.n_rows);
}

// One workgroup of the ASSEMBLE gather (bx: its index among the gather's workgroups).  INLINE:
// the rows are resolved here from the plan instead of read from the row table.
template <int ESZ, bool INLINE>
__device__ __forceinline__ void paged_move_block(const KPagedParams& P, const PlanView& V, int plane, int32_t bx,
                                                 int32_t lgroup, KCosSin* lcs) {
    const KPlane& pl = P.planes[plane];
    const int32_t tb = bx * PAGED_TPB;
    if (int64_t(tb) >= int64_t(P.n_rows) * pl.tpr) return;            // past this plane
    const int32_t t = tb + int32_t(threadIdx.x);
    int32_t i, u;
    row_unit(pl, true, t, P.n_rows, i, u);
    KRowMove e{KROW_SKIP, 0, 0, 0, -1, -1};
    if (i < P.n_rows) e = INLINE ? row_entry(P, V, i) : P.rows[i];
    const bool active = e.src_page != KROW_SKIP;
    // the cos/sin block of the workgroup's first row's shift, fetched before the data loads
    int32_t cs0 = -1;
    if (pl.rot != KROT_NONE) {
        const int32_t i0 = fdiv(tb, pl.tpr_div);
        cs0 = INLINE ? row_entry(P, V, i0).cs : P.rows[i0].cs;
    }
    const CsReg c = cs_fetch(V.cs, cs0 + pl.cs_off, cs0 >= 0 ? pl.n_pairs : 0);
    // PAGED_LPT consecutive layers per thread: one row entry, all loads in flight before any store.
    const int layer0 = lgroup * PAGED_LPT;
    const int nl = min(PAGED_LPT, P.n_layers - layer0);
    const char* src;
    int64_t src_step;
    if (e.src_page == KROW_STUB) {
        // fields read through the entry's address: a copy of the entry indexed by a run-time
        // plane would be placed in LDS, 64 bytes per thread, by the compiler
        const KDirEntry* D = V.dirs + e.dir;
        src_step = D->stub_len * pl.row_bytes;
        src = D->stub[plane] + int64_t(layer0) * src_step + int64_t(e.src_row) * pl.row_bytes;
    } else {
        src_step = pl.layer_stride;
        src = pl.base + int64_t(layer0) * pl.layer_stride + int64_t(e.src_page) * pl.page_stride +
              int64_t(e.src_row) * pl.token_stride;
    }
    char* dst = pl.base + int64_t(layer0) * pl.layer_stride + int64_t(e.dst_page) * pl.page_stride +
                int64_t(e.dst_row) * pl.token_stride;
    const int32_t cs = e.cs >= 0 ? e.cs + pl.cs_off : -1;
    if (pl.rot == KROT_NEOX && !pl.neox_lanes) {        // two-chunk units (rare layouts)
        if (active)
            for (int l = 0; l < nl; ++l)
                move_row_unit<ESZ>(pl, src + l * src_step, dst + l * pl.layer_stride, u, V.cs, cs);
        return;
    }
    const int64_t off = int64_t(u) * 16;
    u32x4 v[PAGED_LPT];
    if (active) {
#pragma unroll
        for (int l = 0; l < PAGED_LPT; ++l)
            if (l < nl) v[l] = ld16(src + l * src_step + off);
    }
    cs_commit(lcs, c, cs0 >= 0 ? pl.n_pairs : 0);
    __syncthreads();
    if (!active) return;
    const bool rot = cs >= 0 && pl.rot != KROT_NONE;
#pragma unroll
    for (int l = 0; l < PAGED_LPT; ++l) {
        if (l < nl) {
            if (rot) {
                if (e.cs == cs0) rotate_chunk<ESZ>(pl, v[l], u, lcs, 0);
                else rotate_chunk<ESZ>(pl, v[l], u, V.cs, cs);
            }
            st16(dst + l * pl.layer_stride + off, v[l]);
        }
    }
}

// One workgroup of the REMAP rotation: band units of all valid rows of all REMAP pages laid end
// to end, PAGED_LPT layers per thread, rotated in place.  The workgroup stages the cos/sin block
// of its first page's shift in LDS; rows with another shift (where runs meet) read the plan's
// table.
template <int ESZ>
__device__ __forceinline__ void paged_remap_block(const KPagedParams& P, const PlanView& V, int plane, int32_t bx,
                                                  int32_t lgroup, KCosSin* lcs) {
    const KPlane& pl = P.planes[plane];
    const int32_t upp = P.page_size * pl.rot_tpr;
    const int32_t tb = bx * PAGED_TPB;
    if (int64_t(tb) >= int64_t(P.n_remap) * upp) return;               // past this plane
    const int32_t t = tb + int32_t(threadIdx.x);
    const int32_t m = fdiv(t, P.remap_div[plane]);
    // the run of the block's first page (block-uniform; a single run comes with the parameters);
    // a lane whose page lies past that run looks its own run up.  With the pages in physical
    // order, each lane reads its resolved page instead.
    KPageRun R0 = P.remap0;
    int32_t next0 = INT32_MAX, cs0 = P.remap0_cs, len0 = P.remap0_len;
    if (P.remap_sorted) {
        // one run: its shift comes with the parameters, no load of the sorted table before the
        // cos/sin fetch
        cs0 = P.n_remap_runs == 1 ? P.remap0_cs : P.remap_sorted[fdiv(tb, P.remap_div[plane])].cs;
    } else if (P.n_remap_runs > 1) {
        const int32_t r0 = run_of(V.remap_runs, P.n_remap_runs, fdiv(tb, P.remap_div[plane]));
        R0 = V.remap_runs[r0];
        next0 = r0 + 1 < P.n_remap_runs ? V.remap_runs[r0 + 1].ord0 : INT32_MAX;
        cs0 = V.dirs[R0.dir].cs;
        len0 = V.seqs[R0.seq].new_len;
    }
    const CsReg c = cs_fetch(V.cs, cs0 + pl.cs_off, cs0 >= 0 ? pl.n_pairs : 0);
    bool active = m < P.n_remap;
    KRemapPage e{0, -1, 0, 0};
    if (active) {
        if (P.remap_sorted) {
            e = P.remap_sorted[m];
        } else if (m < next0) {
            e = remap_entry(P, R0, cs0, len0, m);
        } else {
            const KPageRun R = V.remap_runs[run_of(V.remap_runs, P.n_remap_runs, m)];
            e = remap_entry(P, R, V.dirs[R.dir].cs, V.seqs[R.seq].new_len, m);
        }
    }
    const int32_t f = t - m * upp;
    const int32_t r = fdiv(f, P.rot_div[plane]);
    active = active && r < e.rows;
    const int layer0 = lgroup * PAGED_LPT;
    const int nl = min(PAGED_LPT, P.n_layers - layer0);
    char* row = pl.base + int64_t(layer0) * pl.layer_stride + int64_t(e.page) * pl.page_stride +
                int64_t(r) * pl.token_stride;
    const BandPos bp = band_pos(pl, f - r * pl.rot_tpr);
    u32x4 x[PAGED_LPT], y[PAGED_LPT];
    if (active) band_load(bp, row, pl.layer_stride, nl, x, y);
    cs_commit(lcs, c, cs0 >= 0 ? pl.n_pairs : 0);
    __syncthreads();
    if (!active) return;
    if (e.cs == cs0) band_rotate_store<ESZ>(pl, bp, row, pl.layer_stride, nl, x, y, lcs, 0);
    else band_rotate_store<ESZ>(pl, bp, row, pl.layer_stride, nl, x, y, V.cs, e.cs + pl.cs_off);
}

// One dimension of workgroups: the gather workgroups of every layer group first (plane by plane
// within a layer group), then (small gathers) the workgroups that write the block tables and the
// freed list, then the REMAP workgroups of every layer group (plane by plane).  The gather's and
// the tables' lookup chains are the longest, so they start first and the bulk of a token-slot
// splice (the REMAP rotation) follows; planes without work get no workgroups.  SOLO: only plane 0
// has work in this launch, so no workgroup looks its plane up.  INLINE: the gather resolves its
// rows (no row table) and the launch may carry table work.
template <int ESZ, bool SOLO, bool INLINE>
__global__ __launch_bounds__(PAGED_TPB) void paged_data_kernel(const KPagedParams P) {
    __shared__ KCosSin lcs[KMAX_CS];
    const PlanView V = plan_view(P);
    int32_t b = int32_t(blockIdx.x);
    const int32_t moves = SOLO ? P.move_base[1] : P.move_base[P.n_planes];
    if (b < moves * P.layer_groups) {
        if (P.gather_split) b = xcd_eighth(b, moves * P.layer_groups);
        const int32_t y = fdiv(b, P.move_blk_div);
        const int32_t bx = b - y * moves;
        const int p = SOLO ? 0 : plane_of(P.move_base, P.n_planes, bx);
        paged_move_block<ESZ, INLINE>(P, V, p, bx - P.move_base[p], y, lcs);
        return;
    }
    b -= moves * P.layer_groups;
    if (INLINE) {
        if (b < P.table_blocks) {
            table_work(P, V, int64_t(b) * PAGED_TPB + threadIdx.x);
            return;
        }
        b -= P.table_blocks;
    }
    const int32_t remaps = SOLO ? P.remap_base[1] : P.remap_base[P.n_planes];
    const int32_t y = fdiv(b, P.remap_blk_div);
    const int32_t bx = b - y * remaps;
    const int p = SOLO ? 0 : plane_of(P.remap_base, P.n_planes, bx);
    paged_remap_block<ESZ>(P, V, p, bx - P.remap_base[p], y, lcs);
}

// -------------------------------------------------------------------------- host launchers ---

namespace {

thread_local hipError_t g_last_hip_error = hipSuccess;

int hip_status(hipError_t e) {
    if (e == hipSuccess) return LEYLINE_OK;
    g_last_hip_error = e;
    return LEYLINE_E_HIP;
}

// Launch and report the launch's own status: an error left behind by an earlier, unrelated
// runtime call on this thread is cleared first so it is not blamed on this launch.
template <typename K, typename A>
int launch(K kernel, dim3 grid, hipStream_t stream, const A& args, int block = TPB) {
    (void)hipGetLastError();
    hipLaunchKernelGGL(kernel, grid, dim3(block), 0, stream, args);
    return hip_status(hipGetLastError());
}

int64_t abs64(int64_t v) { return v < 0 ? -v : v; }

// A device buffer given to a call: start and length in bytes (null or empty: no buffer).
struct Span {
    const void* p;
    int64_t bytes;
};

// Whether two of the buffers share a byte.
bool any_overlap(const Span* b, size_t n) {
    for (size_t i = 0; i < n; ++i)
        for (size_t j = i + 1; j < n; ++j) {
            if (!b[i].p || !b[j].p || b[i].bytes <= 0 || b[j].bytes <= 0) continue;
            const uintptr_t a0 = reinterpret_cast<uintptr_t>(b[i].p), c0 = reinterpret_cast<uintptr_t>(b[j].p);
            if (a0 < c0 + uintptr_t(b[j].bytes) && c0 < a0 + uintptr_t(b[i].bytes)) return true;
        }
    return false;
}

}  // namespace

}  // namespace leyline

using namespace leyline;

extern "C" int leyline_pair_bits(void) { return int(sizeof(kcs_t) * 8); }

extern "C" const char* leyline_last_hip_error(void) {
    return hipGetErrorString(g_last_hip_error);
}

// The launch a contiguous job goes to: replacement copies share the round kernel's launches.
static int launch_kind(int kind) { return kind == KJOB_STUB ? int(KJOB_ROUND) : kind; }

// Kernel launches of a schedule (only the ordered-tile launches when tiles_only): with tiles, the
// prep launches and the tile launches; otherwise, per group of independent jobs, one launch per
// job kind present, split further when a launch would exceed its item or cos/sin capacity.
static int contig_launch_count(const leyline_cache* cache, const ContigSchedule& sched, int n_planes,
                               bool tiles_only = false) {
    if (sched.tiles) {
        const int tile = int(sched.tile_launches.size());
        if (tiles_only) return tile;
        const int prep = std::max<int>(1, int((sched.cs.size() + KPREP_CS - 1) / KPREP_CS));
        return prep + tile;
    }
    if (tiles_only) return 0;
    const int32_t cs_need = cos_sin_per_shift(cache);
    int n = 0;
    for (const auto& group : sched.launches)
        for (int kind : {int(KJOB_CHAIN), int(KJOB_ROUND)}) {
            int items = 0, cs = 0;
            bool open = false;
            for (const ContigJobHost& j : group) {
                if (launch_kind(j.kind) != kind) continue;
                const int need = j.kind != KJOB_STUB ? cs_need : 0;
                if (open && (items + n_planes > KMAX_LAUNCH_ITEMS || cs + need > KMAX_CS)) {
                    ++n;
                    items = cs = 0;
                }
                open = true;
                items += n_planes;
                cs += need;
            }
            if (open) ++n;
        }
    return n;
}

// Workgroups of a tile launch: persistent workgroups take tickets until they run out, so the grid
// is the number that can be resident on the device at once (queried once per kernel variant and
// device); more would only start once the tickets are gone.
static int64_t tile_grid_cap(void (*kernel)(KTileParams)) {
    static std::mutex mu;
    static std::vector<std::pair<std::pair<void*, int>, int64_t>> known;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return INT32_MAX;
    std::lock_guard<std::mutex> lock(mu);
    for (const auto& k : known)
        if (k.first.first == reinterpret_cast<void*>(kernel) && k.first.second == dev) return k.second;
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, KTILE_TPB, 0) != hipSuccess ||
        cus <= 0 || per_cu <= 0)
        return INT32_MAX;
    const int64_t cap = int64_t(cus) * per_cu;
    known.push_back({{reinterpret_cast<void*>(kernel), dev}, cap});
    return cap;
}

// The prep launches and ordered-tile launches of a tile schedule.
static int launch_tiles(const leyline_cache* cache, const ContigSchedule& sched, const KPlane* planes,
                        int n_planes, char* ws, int32_t* status, hipStream_t s) {
    // prep: clear the counters and flags, then write the cos/sin table in pieces that fit the
    // kernel arguments
    const int64_t words = sched.ws_cs / 4;
    size_t c = 0;
    do {
        KPrepParams Q;
        std::memset(&Q, 0, sizeof(Q));
        Q.zero = c == 0 ? reinterpret_cast<int32_t*>(ws) : nullptr;
        Q.n_zero = c == 0 ? words : 0;
        const size_t n = std::min<size_t>(sched.cs.size() - c, size_t(KPREP_CS));
        Q.cs_dst = reinterpret_cast<KCosSin*>(ws + sched.ws_cs) + c;
        Q.n_cs = int32_t(n);
        std::copy(sched.cs.begin() + int64_t(c), sched.cs.begin() + int64_t(c + n), Q.cs);
        const int64_t work = std::max<int64_t>(Q.n_zero, Q.n_cs);
        const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((work + TPB - 1) / TPB, 1024));
        const int rc = launch(tile_prep_kernel, dim3(unsigned(blocks)), s, Q);
        if (rc) return rc;
        c += n;
    } while (c < sched.cs.size());
    const bool bf = cache->dtype == LEYLINE_BF16;
    for (size_t k = 0; k < sched.tile_launches.size(); ++k) {
        const TileLaunchHost& tl = sched.tile_launches[k];
        KTileParams P;
        std::memset(&P, 0, sizeof(P));
        std::memcpy(P.planes, planes, sizeof(KPlane) * size_t(n_planes));
        std::copy(tl.items.begin(), tl.items.end(), P.items);
        P.n_items = int32_t(tl.items.size());
        tile_fill_ticket_table(P);
        P.n_tickets = int32_t(tl.tickets);
        P.counter = reinterpret_cast<int32_t*>(ws + 256 * int64_t(k));
        P.flags = reinterpret_cast<int32_t*>(ws + sched.ws_flags);
        P.cs = reinterpret_cast<const KCosSin*>(ws + sched.ws_cs);
        P.status = status;
        using K = void (*)(KTileParams);
        static const K kernels[2][3] = {
            {contig_tile_kernel<4, KROT_NONE>, contig_tile_kernel<4, KROT_INTERLEAVED>, contig_tile_kernel<4, KROT_NEOX>},
            {contig_tile_kernel<2, KROT_NONE>, contig_tile_kernel<2, KROT_INTERLEAVED>, contig_tile_kernel<2, KROT_NEOX>}};
        const K kernel = kernels[bf][launch_rot_style(P)];
        const dim3 grid(static_cast<unsigned>(std::min<int64_t>(tl.tickets, tile_grid_cap(kernel))), 1, 1);
        const int r = launch(kernel, grid, s, P, KTILE_TPB);
        if (r) return r;
    }
    return LEYLINE_OK;
}

extern "C" int leyline_contig_query(const leyline_cache* cache, int64_t seq_len,
                                    const leyline_directive* dirs, int32_t n_dirs,
                                    int64_t* new_len_out, int32_t* n_launches_out,
                                    int32_t* n_tile_launches_out, int64_t* workspace_bytes_out) {
    ContigSchedule sched;
    int rc = plan_contig(cache, seq_len, dirs, n_dirs, &sched);
    if (rc) return rc;
    if (new_len_out) *new_len_out = sched.new_len;
    if (n_launches_out) *n_launches_out = contig_launch_count(cache, sched, cache->n_planes);
    if (n_tile_launches_out) *n_tile_launches_out = contig_launch_count(cache, sched, cache->n_planes, true);
    if (workspace_bytes_out) *workspace_bytes_out = sched.ws_bytes;
    return LEYLINE_OK;
}

// The launches of a planned contiguous splice, on a workspace already checked against the plan.
static int splice_contig_planned(const leyline_cache* cache, const ContigSchedule& sched,
                                 const leyline_directive* dirs, int64_t* new_len_out,
                                 int32_t* device_status, char* ws, hipStream_t s) {
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    int rc = describe_cache(cache, false, planes, &n_planes);
    if (rc) return rc;
    if (sched.tiles) {
        rc = launch_tiles(cache, sched, planes, n_planes, ws, device_status, s);
        if (rc) return rc;
        if (new_len_out) *new_len_out = sched.new_len;
        return LEYLINE_OK;
    }
    // whether a (job, plane) item rotates (it then gets a cos/sin block: KItem::cs >= 0), and its
    // threads; every count must fit a 31-bit index
    const int32_t cs_need = cos_sin_per_shift(cache);
    auto item_rotates = [&](const ContigJobHost& j, int p) {
        return j.kind != KJOB_STUB && cs_need > 0 && planes[p].rot != KROT_NONE;
    };
    auto item_threads = [&](const ContigJobHost& j, int p) -> int64_t {
        if (j.kind == KJOB_CHAIN) return std::min<int64_t>(j.count, abs64(j.delta)) * planes[p].units_all;
        const int rpt = round_rows_per_thread(item_rotates(j, p));
        return (j.count + rpt - 1) / rpt * planes[p].tpr;
    };
    for (const auto& jobs : sched.launches)
        for (const auto& j : jobs)
            for (int p = 0; p < n_planes; ++p)
                if (item_threads(j, p) > INT32_MAX - TPB) return LEYLINE_E_INVAL;
    for (const auto& group : sched.launches) {
        // the jobs of a group are independent; replacement copies, chains and rounds go to
        // separate launches, each a list of (job, plane) items selected by blockIdx.z
        for (int kind : {int(KJOB_CHAIN), int(KJOB_ROUND)}) {
            // ROUND launches carry the group's rounds and replacement copies, each (job, plane)
            // item with its own range of workgroups; CHAIN launches select items by blockIdx.z
            KContigParams P;
            std::vector<KCosSin> cs;
            int64_t max_blocks = 0, total_blocks = 0;
            auto flush = [&]() -> int {
                if (P.n_items == 0) return LEYLINE_OK;
                if (cs.size() > size_t(KMAX_CS) || max_blocks > INT32_MAX || total_blocks > INT32_MAX)
                    return LEYLINE_E_INVAL;
                std::copy(cs.begin(), cs.end(), P.cs);
                for (int32_t i = P.n_items; i < KMAX_LAUNCH_ITEMS; ++i) P.block0[i] = INT32_MAX;
                int r;
                if (kind == KJOB_CHAIN) {
                    const dim3 grid(unsigned(max_blocks), unsigned(cache->n_layers), unsigned(P.n_items));
                    r = cache->dtype == LEYLINE_BF16 ? launch(contig_chain_kernel<2>, grid, s, P)
                                                     : launch(contig_chain_kernel<4>, grid, s, P);
                } else {
                    const dim3 grid(unsigned(total_blocks), unsigned(cache->n_layers), 1);
                    r = cache->dtype == LEYLINE_BF16 ? launch(contig_move_kernel<2>, grid, s, P, MOVE_TPB)
                                                     : launch(contig_move_kernel<4>, grid, s, P, MOVE_TPB);
                }
                P.n_items = 0;
                cs.clear();
                max_blocks = total_blocks = 0;
                return r;
            };
            std::memset(&P, 0, sizeof(P));
            for (const ContigJobHost& j : group) {
                if (launch_kind(j.kind) != kind) continue;
                const int32_t need = j.kind != KJOB_STUB ? cs_need : 0;
                if (P.n_items + n_planes > KMAX_LAUNCH_ITEMS || int32_t(cs.size()) + need > KMAX_CS) {
                    rc = flush();
                    if (rc) return rc;
                }
                const int32_t cs0 = (j.kind != KJOB_STUB && cs_need > 0) ? append_cos_sin(cache, j.delta, cs) : -1;
                for (int p = 0; p < n_planes; ++p) {
                    const int64_t th = item_threads(j, p);
                    if (th == 0) continue;
                    KItem& it = P.items[P.n_items];
                    std::memset(&it, 0, sizeof(it));
                    it.pl = planes[p];
                    it.src0 = j.src0;
                    it.dst0 = j.dst0;
                    it.count = j.count;
                    it.delta = j.delta;
                    it.kind = j.kind;
                    it.chains = int32_t(kind == KJOB_CHAIN ? std::min<int64_t>(j.count, abs64(j.delta)) : 0);
                    it.cs = item_rotates(j, p) ? cs0 + planes[p].cs_off : -1;
                    if (j.kind == KJOB_STUB) it.stub = static_cast<const char*>(dirs[j.dir].stub[p]);
                    const int block = kind == KJOB_CHAIN ? TPB : MOVE_TPB;
                    const int64_t blocks = (th + block - 1) / block;
                    P.block0[P.n_items] = int32_t(std::min<int64_t>(total_blocks, INT32_MAX));
                    max_blocks = std::max(max_blocks, blocks);
                    total_blocks += blocks;
                    ++P.n_items;
                }
            }
            rc = flush();
            if (rc) return rc;
        }
    }
    if (new_len_out) *new_len_out = sched.new_len;
    return LEYLINE_OK;
}

extern "C" int leyline_splice_contig(const leyline_cache* cache, int64_t seq_len,
                                     const leyline_directive* dirs, int32_t n_dirs,
                                     int64_t* new_len_out, int32_t* device_status,
                                     void* workspace, int64_t workspace_bytes, void* stream) {
    ContigSchedule sched;
    int rc = plan_contig(cache, seq_len, dirs, n_dirs, &sched);
    if (rc) return rc;
    if (sched.ws_bytes > 0 && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) ||
                               workspace_bytes < sched.ws_bytes))
        return LEYLINE_E_WORKSPACE;
    return splice_contig_planned(cache, sched, dirs, new_len_out, device_status, static_cast<char*>(workspace),
                                 static_cast<hipStream_t>(stream));
}

// ------------------------------------------------------------- splice without allocation ---
//
// The contiguous splice's workspace for callers that cannot allocate device memory (graph
// capture, serving loops, harnesses that forbid hipMalloc): a fixed array in device memory, one
// copy per GPU, held until the process ends.  Host code never passes the array's name (a host
// stand-in, not a device address): its device address is looked up once per device, with that
// device current, and only that address is handed to kernels.
static __device__ __align__(256) char scratch[LEYLINE_SCRATCH_BYTES];

namespace {

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices];

// The scratch array's address on the calling thread's current device; the stream must run on
// that device.
int scratch_on_current_device(hipStream_t stream, char** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e);
    if (dev < 0 || dev >= kScratchDevices) return LEYLINE_E_INVAL;
    if (stream) {
        hipDevice_t sd = -1;
        e = hipStreamGetDevice(stream, &sd);
        if (e != hipSuccess) return hip_status(e);
        if (sd != dev) return LEYLINE_E_INVAL;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(e);
        if (!p) return LEYLINE_E_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = static_cast<char*>(g_scratch_ptr[dev]);
    return LEYLINE_OK;
}

}  // namespace

extern "C" int leyline_splice_contig_noalloc(const leyline_cache* cache, int64_t seq_len,
                                             const leyline_directive* dirs, int32_t n_dirs,
                                             int64_t* new_len_out, int32_t* device_status, void* stream) {
    ContigSchedule sched;
    int rc = plan_contig(cache, seq_len, dirs, n_dirs, &sched);
    if (rc) return rc;
    if (sched.ws_bytes > LEYLINE_SCRATCH_BYTES) return LEYLINE_E_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* ws = nullptr;
    if (sched.ws_bytes > 0) {
        rc = scratch_on_current_device(s, &ws);
        if (rc) return rc;
    }
    return splice_contig_planned(cache, sched, dirs, new_len_out, device_status, ws, s);
}

// The rotation kernel variant for (dtype, one plane only, paged cache).
static int launch_rotate(bool bf16, bool solo, bool paged, dim3 grid, hipStream_t s, const KRotateParams& P) {
    using K = void (*)(KRotateParams);
    static const K table[2][2][2] = {
        {{rotate_rows_kernel<4, false, false>, rotate_rows_kernel<4, false, true>},
         {rotate_rows_kernel<4, true, false>, rotate_rows_kernel<4, true, true>}},
        {{rotate_rows_kernel<2, false, false>, rotate_rows_kernel<2, false, true>},
         {rotate_rows_kernel<2, true, false>, rotate_rows_kernel<2, true, true>}}};
    return launch(table[bf16][solo][paged], grid, s, P, PAGED_TPB);
}

extern "C" int leyline_rotate_delta(const leyline_cache* cache, int64_t delta,
                                    const int64_t* rows, int64_t row0, int64_t n_rows,
                                    int32_t* device_status, void* stream) {
    if (!cache) return LEYLINE_E_INVAL;
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    const bool paged = cache->page_size > 0;
    int rc = describe_cache(cache, paged, planes, &n_planes);
    if (rc) return rc;
    if (n_rows < 0) return LEYLINE_E_INVAL;
    const int64_t total_rows = paged ? cache->capacity * cache->page_size : cache->capacity;
    if (!rows && (row0 < 0 || row0 > total_rows || n_rows > total_rows - row0)) return LEYLINE_E_RANGE;
    if (n_rows == 0 || delta == 0) return LEYLINE_OK;   // R(0) is the identity
    if (paged && total_rows > INT32_MAX) return LEYLINE_E_INVAL;
    KRotateParams P;
    std::memset(&P, 0, sizeof(P));
    int32_t max_rot = 0;
    for (int p = 0; p < n_planes; ++p) {
        max_rot = std::max(max_rot, planes[p].rot_tpr);
        P.rot_div[p] = make_div(std::max(1, planes[p].rot_tpr));
        if (n_rows * planes[p].rot_tpr > INT32_MAX - 1024) return LEYLINE_E_INVAL;
    }
    if (max_rot == 0) return LEYLINE_OK;
    std::memcpy(P.planes, planes, sizeof(planes));
    P.h.n_planes = n_planes;
    P.h.n_layers = cache->n_layers;
    P.h.page_size = paged ? cache->page_size : 0;
    P.page_div = make_div(paged ? cache->page_size : 1);
    P.h.total_rows = total_rows;
    P.h.rows = rows;
    P.h.row0 = row0;
    P.h.n_rows = n_rows;
    P.h.status = device_status;
    std::vector<KCosSin> cs;
    append_cos_sin(cache, delta, cs);
    std::copy(cs.begin(), cs.end(), P.cs);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bf16 = cache->dtype == LEYLINE_BF16;
    // one launch: the workgroups of each rotary plane after those of the previous one
    int64_t total = 0;
    P.rot_base[0] = 0;
    for (int p = 0; p < n_planes; ++p) {
        if (planes[p].rot_tpr > 0) total += (n_rows * planes[p].rot_tpr + PAGED_TPB - 1) / PAGED_TPB;
        if (total > INT32_MAX - 1024) return LEYLINE_E_INVAL;
        P.rot_base[p + 1] = int32_t(total);
    }
    const dim3 grid(unsigned(total), unsigned((cache->n_layers + PAGED_LPT - 1) / PAGED_LPT), 1);
    const bool solo = P.rot_base[1] == total;                            // plane 0 only
    rc = launch_rotate(bf16, solo, paged, grid, s, P);
    if (rc) return rc;
    return LEYLINE_OK;
}

// The paged data kernel variant for (dtype, one plane only, inline rows).
static int launch_paged_data(bool bf16, bool solo, bool inl, dim3 grid, hipStream_t s, const KPagedParams& P) {
    using K = void (*)(KPagedParams);
    static const K table[2][2][2] = {
        {{paged_data_kernel<4, false, false>, paged_data_kernel<4, false, true>},
         {paged_data_kernel<4, true, false>, paged_data_kernel<4, true, true>}},
        {{paged_data_kernel<2, false, false>, paged_data_kernel<2, false, true>},
         {paged_data_kernel<2, true, false>, paged_data_kernel<2, true, true>}}};
    return launch(table[bf16][solo][inl], grid, s, P, PAGED_TPB);
}

extern "C" int leyline_splice_paged(const leyline_cache* cache, int32_t n_seqs, const int32_t* seq_lens,
                                    const int32_t* block_table_in, int32_t* block_table_out, int32_t bt_stride,
                                    const leyline_directive* dirs, int32_t n_dirs, uint32_t flags,
                                    const int32_t* free_pages, int32_t n_free,
                                    int32_t* freed_pages_out, int32_t freed_cap,
                                    int32_t* new_seq_lens_out, int32_t* n_fresh_used_out, int32_t* n_freed_out,
                                    int32_t* device_status,
                                    void* workspace, int64_t workspace_bytes, void* stream) {
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    int rc = describe_cache(cache, true, planes, &n_planes);
    if (rc) return rc;
    // bt_stride 0 (tables without columns) suits only sequences that stay empty, which the
    // table-width check below enforces, as leyline_paged_query's does
    if (bt_stride < 0 || n_free < 0 || freed_cap < 0 || workspace_bytes < 0) return LEYLINE_E_INVAL;
    const int64_t bt_bytes = int64_t(n_seqs > 0 ? n_seqs : 0) * bt_stride * 4;
    if (bt_bytes > 0 && (!block_table_in || !block_table_out || block_table_in == block_table_out))
        return LEYLINE_E_INVAL;
    if (flags & ~uint32_t(LEYLINE_PAGED_COPY_ON_WRITE)) return LEYLINE_E_INVAL;
    {
        // One launch reads the old tables and the free list while it writes the new tables, the
        // freed list, the workspace and the status word: no two of these may share a byte.
        const Span bufs[] = {{block_table_in, bt_bytes},    {block_table_out, bt_bytes},
                             {free_pages, int64_t(n_free) * 4}, {freed_pages_out, int64_t(freed_cap) * 4},
                             {workspace, workspace_bytes},  {device_status, 4}};
        if (any_overlap(bufs, sizeof(bufs) / sizeof(bufs[0]))) return LEYLINE_E_INVAL;
    }
    PagedPlan plan;
    rc = plan_paged(cache->page_size, n_seqs, seq_lens, dirs, n_dirs, n_planes,
                    !(flags & LEYLINE_PAGED_COPY_ON_WRITE), &plan);
    if (rc) return rc;
    rc = check_table_width(plan, seq_lens, bt_stride);
    if (rc) return rc;
    if (plan.n_fresh > n_free) return LEYLINE_E_CAPACITY;
    if (plan.n_freed > freed_cap) return LEYLINE_E_CAPACITY;
    if (plan.n_fresh > 0 && !free_pages) return LEYLINE_E_INVAL;
    if (plan.n_freed > 0 && !freed_pages_out) return LEYLINE_E_INVAL;
    PagedImage img;
    rc = build_paged_image(cache, plan, n_seqs, plan.dirs, n_dirs, bt_stride, &img);
    if (rc) return rc;
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < img.tables.total)
        return LEYLINE_E_WORKSPACE;

    hipStream_t s = static_cast<hipStream_t>(stream);
    const KPagedTables& t = img.tables;
    char* ws = static_cast<char*>(workspace);
    if (int64_t(t.n_rows) + t.n_remap > INT32_MAX - 1024) return LEYLINE_E_INVAL;
    const bool row_table = t.n_rows > KINLINE_ROWS;       // else the gather resolves its rows
    for (int p = 0; p < n_planes; ++p) {
        if (int64_t(t.n_rows) * planes[p].tpr > INT32_MAX - 1024) return LEYLINE_E_INVAL;
        if (int64_t(t.n_remap) * cache->page_size * planes[p].rot_tpr > INT32_MAX - 1024) return LEYLINE_E_INVAL;
    }
    if (t.upload > INT32_MAX) return LEYLINE_E_INVAL;
    const bool inline_plan = t.upload <= KPLAN_INLINE;
    if (!inline_plan) {
        rc = hip_status(hipMemcpyAsync(ws, img.bytes.data(), size_t(t.upload), hipMemcpyHostToDevice, s));
        if (rc) return rc;
    }
    const int64_t n_table = int64_t(n_seqs) * bt_stride;
    const int64_t n_tables = n_table + t.n_freed;          // block-table and freed-list entries
    if (int64_t(t.n_rows) + n_tables > INT32_MAX - 1024) return LEYLINE_E_INVAL;
    if (int64_t(t.n_rows) + t.n_remap + n_tables > 0) {
        KPagedParams P;
        std::memset(&P, 0, sizeof(P));
        std::memcpy(P.planes, planes, sizeof(planes));
        P.n_planes = n_planes;
        P.n_layers = cache->n_layers;
        P.page_size = cache->page_size;
        P.bt_stride = bt_stride;
        P.n_asm = t.n_asm;
        P.n_remap = t.n_remap;
        P.n_rows = t.n_rows;
        int32_t max_tpr = 1, max_upp = 1;
        for (int p = 0; p < n_planes; ++p) {
            const int32_t upp = cache->page_size * planes[p].rot_tpr;
            max_tpr = std::max(max_tpr, planes[p].tpr);
            max_upp = std::max(max_upp, upp);
            P.remap_div[p] = make_div(std::max(1, upp));
            P.rot_div[p] = make_div(std::max(1, planes[p].rot_tpr));
        }
        P.capacity = cache->capacity;
        // a plan small enough travels in the kernel arguments; otherwise it was uploaded above
        P.plan = inline_plan ? nullptr : ws;
        if (inline_plan) std::memcpy(P.blob, img.bytes.data(), size_t(t.upload));
        P.off_seq = int32_t(t.off_seq);
        P.off_dir = int32_t(t.off_dir);
        P.off_cs = int32_t(t.off_cs);
        P.off_runs = int32_t(t.off_runs);
        P.off_asm_runs = int32_t(t.off_asm_runs);
        P.off_remap_runs = int32_t(t.off_remap_runs);
        P.off_freed_runs = int32_t(t.off_freed_runs);
        P.n_asm_runs = t.n_asm_runs;
        P.n_remap_runs = t.n_remap_runs;
        P.rows = row_table ? reinterpret_cast<KRowMove*>(ws + t.off_rows) : nullptr;
        if (t.n_remap_runs == 1) {
            // the single REMAP run, its shift's cos/sin entry and its sequence's new length
            std::memcpy(&P.remap0, img.bytes.data() + t.off_remap_runs, sizeof(KPageRun));
            KDirEntry d;
            std::memcpy(&d, img.bytes.data() + t.off_dir + int64_t(P.remap0.dir) * int64_t(sizeof(KDirEntry)), sizeof(d));
            KSeqEntry q;
            std::memcpy(&q, img.bytes.data() + t.off_seq + int64_t(P.remap0.seq) * int64_t(sizeof(KSeqEntry)), sizeof(q));
            P.remap0_cs = d.cs;
            P.remap0_len = q.new_len;
        }
        P.bt_out = block_table_out;
        P.freed_out = freed_pages_out;
        P.n_table = int32_t(n_table);
        P.n_freed = t.n_freed;
        P.n_freed_runs = t.n_freed_runs;
        P.bt_in = block_table_in;
        P.free_pages = free_pages;
        P.n_free = n_free;
        P.status = device_status;
        const bool bf16 = cache->dtype == LEYLINE_BF16;
        const unsigned layer_groups = unsigned((cache->n_layers + PAGED_LPT - 1) / PAGED_LPT);
        if (row_table) {
            if (t.n_asm >= KORDER_MIN) {
                int32_t shift = 0;
                while (((cache->capacity - 1) >> shift) >= KORDER_BUCKETS) ++shift;
                P.order_shift = shift;
                P.order = reinterpret_cast<int32_t*>(ws + t.off_order);
                rc = launch(paged_order_kernel, dim3(1), s, P, ORDER_TPB);
                if (rc) return rc;
            }
            rc = launch(paged_resolve_kernel, dim3(unsigned((int64_t(t.n_rows) + n_tables + TPB - 1) / TPB)), s, P);
            if (rc) return rc;
        } else {
            // the first data launch writes the tables, spread over its layer groups
            P.table_blocks = int32_t((n_tables + PAGED_TPB - 1) / PAGED_TPB);
        }
        if (t.remap_sorted) {
            // wide rotary bands: the REMAP pages in physical order
            int32_t shift = 0;
            while (((cache->capacity - 1) >> shift) >= KORDER_BUCKETS) ++shift;
            P.remap_shift = shift;
            P.remap_sorted = reinterpret_cast<KRemapPage*>(ws + t.off_remap_sorted);
            // entries pack into 8 bytes: shift index + 1 and valid rows below 2^16
            P.remap_pack = cache->page_size < 65536 && t.n_cs < 65535 ? 1 : 0;
            rc = launch(paged_remap_order_kernel, dim3(1), s, P, ORDER_TPB);
            if (rc) return rc;
        }
        // data kernel, one launch: gather workgroups, then the REMAP workgroups of every rotary
        // plane, then (small gathers) the table work
        int64_t mb = 0, rb = 0;
        P.move_base[0] = P.remap_base[0] = 0;
        for (int p = 0; p < n_planes; ++p) {
            if (t.n_rows > 0) mb += (int64_t(t.n_rows) * planes[p].tpr + PAGED_TPB - 1) / PAGED_TPB;
            if (t.n_remap > 0 && planes[p].rot_tpr > 0)
                rb += (int64_t(t.n_remap) * cache->page_size * planes[p].rot_tpr + PAGED_TPB - 1) / PAGED_TPB;
            if (mb > INT32_MAX - 1024 || rb > INT32_MAX - 1024 || mb + rb > INT32_MAX - 1024)
                return LEYLINE_E_INVAL;
            P.move_base[p + 1] = int32_t(mb);
            P.remap_base[p + 1] = int32_t(rb);
        }
        const int64_t blocks = (mb + rb) * int64_t(layer_groups) + P.table_blocks;
        if (blocks > INT32_MAX - 1024) return LEYLINE_E_INVAL;
        if (blocks > 0) {
            P.layer_groups = int32_t(layer_groups);
            P.gather_split = cache->page_size >= LEYLINE_GATHER_SPLIT_PAGE ? 1 : 0;
            P.move_blk_div = make_div(int32_t(std::max<int64_t>(1, mb)));
            P.remap_blk_div = make_div(int32_t(std::max<int64_t>(1, rb)));
            const bool solo = P.move_base[1] == mb && P.remap_base[1] == rb;   // plane 0 only
            rc = launch_paged_data(bf16, solo, !row_table, dim3(unsigned(blocks)), s, P);
            if (rc) return rc;
        }
    }
    if (new_seq_lens_out)
        for (int32_t b = 0; b < n_seqs; ++b) new_seq_lens_out[b] = plan.new_lens[size_t(b)];
    if (n_fresh_used_out) *n_fresh_used_out = plan.n_fresh;
    if (n_freed_out) *n_freed_out = plan.n_freed;
    return LEYLINE_OK;
}
