// HIP kernels of the KV-cache splice for gfx950 (MI355X), and the C-ABI entry points that
// enqueue them.
//
// The path is bandwidth-bound element movement with a little fp32 arithmetic on the rotary
// band (about 0.1-0.4 flop per byte), so there is no matrix-core work here: rows are moved as
// 16-byte vectors by 64-wide wavefronts, each wave touching whole 128-byte lines, and the
// re-anchoring rotation (Eq. "rotate": each pair (a, b) becomes (a c - b s, a s + b c)) is
// applied in registers between the load and the store of a moved row.  cos/sin of
// (shift * theta_i) come from the host, evaluated in fp64 once per call and shift, and live in
// registers for the whole of a thread's work.
//
// In-place contiguous compaction.  A segment moved left by m rows writes row x with the old
// content of row x + m.  Rows are split into m "chains": chain c owns rows c, c+m, c+2m, ...
// of the segment, and one thread walks its chain in ascending order (descending for a right
// shift), so every row it overwrites is one it has already read itself; different chains and
// different 16-byte columns never touch the same bytes.  Loads of up to WIN consecutive chain
// steps are issued together before their stores, which keeps enough bytes in flight per thread.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "kparams.hpp"
#include "leyline.h"
#include "plan.hpp"

namespace leyline {

constexpr int TPB = 256;
constexpr int WIN = 8;
constexpr int MAX_PAGE = 256;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld16(const char* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(char* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// ----------------------------------------------------------------------- element helpers ---

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest, ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ void rot_pair(float& a, float& b, float c, float s) {
    const float a2 = a * c - b * s;
    const float b2 = a * s + b * c;
    a = a2;
    b = b2;
}

// Elements per 16-byte chunk for an element size.
template <int ESZ> struct Elt { static constexpr int EPC = 16 / ESZ; };

// Rotate one interleaved chunk: EPC/2 pairs (2i, 2i+1).
template <int ESZ> __device__ __forceinline__ void rot_interleaved(u32x4& v, const float* c, const float* s);
template <> __device__ __forceinline__ void rot_interleaved<2>(u32x4& v, const float* c, const float* s) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float a = bf_lo(v[i]), b = bf_hi(v[i]);
        rot_pair(a, b, c[i], s[i]);
        v[i] = f32_to_bf16(a) | (f32_to_bf16(b) << 16);
    }
}
template <> __device__ __forceinline__ void rot_interleaved<4>(u32x4& v, const float* c, const float* s) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        float a = __uint_as_float(v[2 * i]), b = __uint_as_float(v[2 * i + 1]);
        rot_pair(a, b, c[i], s[i]);
        v[2 * i] = __float_as_uint(a);
        v[2 * i + 1] = __float_as_uint(b);
    }
}

// Rotate a half-split (NEOX) chunk pair: element e of the low-half chunk with element e of the
// high-half chunk, EPC pairs.
template <int ESZ> __device__ __forceinline__ void rot_neox(u32x4& va, u32x4& vb, const float* c, const float* s);
template <> __device__ __forceinline__ void rot_neox<2>(u32x4& va, u32x4& vb, const float* c, const float* s) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float a0 = bf_lo(va[i]), a1 = bf_hi(va[i]);
        float b0 = bf_lo(vb[i]), b1 = bf_hi(vb[i]);
        rot_pair(a0, b0, c[2 * i], s[2 * i]);
        rot_pair(a1, b1, c[2 * i + 1], s[2 * i + 1]);
        va[i] = f32_to_bf16(a0) | (f32_to_bf16(a1) << 16);
        vb[i] = f32_to_bf16(b0) | (f32_to_bf16(b1) << 16);
    }
}
template <> __device__ __forceinline__ void rot_neox<4>(u32x4& va, u32x4& vb, const float* c, const float* s) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float a = __uint_as_float(va[i]), b = __uint_as_float(vb[i]);
        rot_pair(a, b, c[i], s[i]);
        va[i] = __float_as_uint(a);
        vb[i] = __float_as_uint(b);
    }
}

// A work unit of a row: chunk a, partner chunk b (-1 if none), first rotary pair, kind.
struct Unit {
    int32_t a, b, pair, kind;   // kind: KROT_NONE / KROT_INTERLEAVED / KROT_NEOX
};

template <int ESZ>
__device__ __forceinline__ Unit map_unit(const KPlane& p, int32_t u) {
    constexpr int EPC = Elt<ESZ>::EPC;
    Unit r{u, -1, 0, KROT_NONE};
    if (p.rot == KROT_INTERLEAVED) {
        const int32_t h = u / p.head_chunks, j = u - h * p.head_chunks;
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
            const int32_t h = u / uh, j = u - h * uh;
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

// A rotary-only unit (the u-th rotary work unit of a row).
template <int ESZ>
__device__ __forceinline__ Unit map_rot_unit(const KPlane& p, int32_t u) {
    constexpr int EPC = Elt<ESZ>::EPC;
    Unit r{0, -1, 0, p.rot};
    if (p.rot == KROT_INTERLEAVED) {
        const int32_t h = u / p.rot_chunks, j = u - h * p.rot_chunks;
        r.a = h * p.head_chunks + p.rot_lo + j;
        r.pair = j * (EPC / 2);
    } else {
        const int32_t half = p.rot_chunks >> 1;
        const int32_t h = u / half, j = u - h * half;
        r.a = h * p.head_chunks + p.rot_lo + j;
        r.b = r.a + half;
        r.pair = j * EPC;
    }
    return r;
}

template <int ESZ>
__device__ __forceinline__ void load_cs(const KCosSin* table, const Unit& un, float* c, float* s) {
    constexpr int EPC = Elt<ESZ>::EPC;
    const int n = un.kind == KROT_NEOX ? EPC : EPC / 2;
#pragma unroll
    for (int i = 0; i < EPC; ++i) {
        if (i < n) {
            const KCosSin v = table[un.pair + i];
            c[i] = v.c;
            s[i] = v.s;
        } else {
            c[i] = 1.0f;
            s[i] = 0.0f;
        }
    }
}

template <int ESZ>
__device__ __forceinline__ void apply_rot(const Unit& un, u32x4& va, u32x4& vb, const float* c, const float* s) {
    if (un.kind == KROT_INTERLEAVED) rot_interleaved<ESZ>(va, c, s);
    else if (un.kind == KROT_NEOX) rot_neox<ESZ>(va, vb, c, s);
}

// --------------------------------------------------------------------- contiguous splice ---

template <int ESZ>
__global__ __launch_bounds__(TPB) void contig_splice_kernel(const KContigParams P) {
    const int layer = blockIdx.y;
    const int bx = blockIdx.x;
    int item = 0;
    while (item < P.n_items - 1 && bx >= P.item_block_end[item]) ++item;
    const int first = item ? P.item_block_end[item - 1] : 0;
    const int pid = P.item_plane[item];
    const KPlane& pl = P.planes[pid];
    const KContigJob& J = P.jobs[P.item_job[item]];
    const int32_t t = (bx - first) * TPB + int32_t(threadIdx.x);
    const int32_t U = pl.units;
    const int32_t c = t / U, u = t - c * U;
    if (c >= J.chains) return;
    const Unit un = map_unit<ESZ>(pl, u);
    const int64_t oa = int64_t(un.a) * 16, ob = int64_t(un.b) * 16;
    char* lbase = pl.base + int64_t(layer) * pl.layer_stride;
    const int64_t ts = pl.token_stride;

    if (J.is_stub) {
        const char* src = J.stub[pid] + (int64_t(layer) * J.count + c) * pl.row_bytes;
        char* dst = lbase + (J.dst0 + c) * ts;
        const u32x4 va = ld16(src + oa);
        u32x4 vb;
        if (un.b >= 0) vb = ld16(src + ob);
        st16(dst + oa, va);
        if (un.b >= 0) st16(dst + ob, vb);
        return;
    }

    float cs_c[Elt<ESZ>::EPC], cs_s[Elt<ESZ>::EPC];
    const bool rot = J.cs >= 0 && un.kind != KROT_NONE;
    if (rot) load_cs<ESZ>(P.cs + J.cs + pl.cs_off, un, cs_c, cs_s);

    const int64_t m = J.delta < 0 ? -J.delta : J.delta;
    const int64_t steps = (J.count - c + m - 1) / m;
    const char* src_c = lbase + (J.src0 + c) * ts;   // step k reads src_c + k*m*ts
    const int64_t step_bytes = m * ts;
    const int64_t dshift = J.delta * ts;             // destination = source + dshift
    const bool down = J.delta < 0;                   // left shift: ascending chain walk

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
                if (rot) apply_rot<ESZ>(un, va[w], vb[w], cs_c, cs_s);
                char* d = const_cast<char*>(src_c) + k * step_bytes + dshift;
                st16(d + oa, va[w]);
                if (un.b >= 0) st16(d + ob, vb[w]);
            }
        }
    }
}

// ------------------------------------------------------------------------ rotate in place ---

template <int ESZ>
__global__ __launch_bounds__(TPB) void rotate_rows_kernel(const KRotateParams P) {
    const int layer = blockIdx.y;
    const int64_t t = int64_t(blockIdx.x) * TPB + threadIdx.x;
    const int64_t i = t / P.units_per_row;
    if (i >= P.n_rows) return;
    int32_t u = int32_t(t - i * P.units_per_row);
    int p = 0;
    while (p < P.n_planes - 1 && u >= P.planes[p].rot_units) {
        u -= P.planes[p].rot_units;
        ++p;
    }
    const KPlane& pl = P.planes[p];
    const int64_t row = P.rows ? P.rows[i] : P.row0 + i;
    if (row < 0 || row >= P.total_rows) {
        if (P.status && u == 0 && p == 0) atomicOr(P.status, int(LEYLINE_STATUS_BAD_ROW));
        return;
    }
    const Unit un = map_rot_unit<ESZ>(pl, u);
    char* r = pl.base + int64_t(layer) * pl.layer_stride;
    if (P.page_size > 0)
        r += (row / P.page_size) * pl.page_stride + (row % P.page_size) * pl.token_stride;
    else
        r += row * pl.token_stride;
    float cs_c[Elt<ESZ>::EPC], cs_s[Elt<ESZ>::EPC];
    load_cs<ESZ>(P.cs + pl.cs_off, un, cs_c, cs_s);
    u32x4 va = ld16(r + int64_t(un.a) * 16), vb;
    if (un.b >= 0) vb = ld16(r + int64_t(un.b) * 16);
    apply_rot<ESZ>(un, va, vb, cs_c, cs_s);
    st16(r + int64_t(un.a) * 16, va);
    if (un.b >= 0) st16(r + int64_t(un.b) * 16, vb);
}

// ------------------------------------------------------------------------------ paged splice ---
//
// One block per (page task, layer, plane).  ASSEMBLE tasks gather the rows of one new page
// (prefix remainder, replacement tokens and shifted downstream rows, possibly from two old
// pages) into a fresh page, rotating downstream rows on the way.  REMAP tasks rotate the
// rotary bands of a re-used page in place.  Nothing is written to an old page except the
// rotary bands of REMAP pages, which no ASSEMBLE task reads.

template <int ESZ>
__global__ __launch_bounds__(TPB) void paged_splice_kernel(const KPagedParams P) {
    __shared__ const char* row_src[MAX_PAGE];
    __shared__ int32_t row_cs[MAX_PAGE];
    __shared__ char* page_dst;
    const int layer = blockIdx.y;
    const int plane = blockIdx.z;
    const KPlane& pl = P.planes[plane];
    const int64_t lbase_off = int64_t(layer) * pl.layer_stride;
    const int task = blockIdx.x;

    if (task < P.n_asm) {
        const KAssembleTask T = P.asm_tasks[task];
        const KSeqEntry S = P.seqs[T.seq];
        const int64_t lo = int64_t(T.k) * P.page_size;
        const int valid = int(min(int64_t(P.page_size), int64_t(S.new_len) - lo));
        if (threadIdx.x == 0) {
            const int32_t fp = T.fresh < P.n_free ? P.free_pages[T.fresh] : -1;
            if (fp < 0 || fp >= P.capacity) {
                if (P.status) atomicOr(P.status, int(LEYLINE_STATUS_BAD_PAGE));
                page_dst = nullptr;
            } else {
                page_dst = pl.base + lbase_off + int64_t(fp) * pl.page_stride;
            }
        }
        for (int r = threadIdx.x; r < valid; r += TPB) {
            const int64_t q = lo + r;
            // last directive of the sequence whose replacement starts at or before q
            int32_t jlo = 0, jhi = S.dir_count;
            while (jlo < jhi) {
                const int32_t mid = (jlo + jhi) >> 1;
                if (P.dirs[S.dir_begin + mid].stub_start <= q) jlo = mid + 1; else jhi = mid;
            }
            int64_t old = q;
            int32_t cs = -1;
            const char* src = nullptr;
            if (jlo > 0) {
                const KDirEntry& D = P.dirs[S.dir_begin + jlo - 1];
                if (q < D.stub_start + D.stub_len) {
                    src = D.stub[plane] + (int64_t(layer) * D.stub_len + (q - D.stub_start)) * pl.row_bytes;
                    old = -1;
                } else {
                    old = q - D.delta;
                    cs = D.cs;
                }
            }
            if (old >= 0) {
                const int32_t pg = P.bt_in[int64_t(T.seq) * P.bt_stride + old / P.page_size];
                if (pg < 0 || pg >= P.capacity) {
                    if (P.status) atomicOr(P.status, int(LEYLINE_STATUS_BAD_PAGE));
                    src = nullptr;
                } else {
                    src = pl.base + lbase_off + int64_t(pg) * pl.page_stride + (old % P.page_size) * pl.token_stride;
                }
            }
            row_src[r] = src;
            row_cs[r] = cs;
        }
        __syncthreads();
        char* dst_page = page_dst;
        if (!dst_page) return;
        const int32_t U = pl.units;
        const int32_t total = valid * U;
        for (int32_t f0 = 0; f0 < total; f0 += TPB * WIN) {
            u32x4 va[WIN], vb[WIN];
            Unit un[WIN];
            int32_t rr[WIN];
#pragma unroll
            for (int w = 0; w < WIN; ++w) {
                const int32_t f = f0 + w * TPB + int32_t(threadIdx.x);
                rr[w] = -1;
                if (f < total) {
                    const int32_t r = f / U;
                    un[w] = map_unit<ESZ>(pl, f - r * U);
                    const char* s = row_src[r];
                    if (s) {
                        rr[w] = r;
                        va[w] = ld16(s + int64_t(un[w].a) * 16);
                        if (un[w].b >= 0) vb[w] = ld16(s + int64_t(un[w].b) * 16);
                    }
                }
            }
#pragma unroll
            for (int w = 0; w < WIN; ++w) {
                const int32_t r = rr[w];
                if (r >= 0) {
                    const int32_t cs = row_cs[r];
                    if (cs >= 0 && un[w].kind != KROT_NONE) {
                        float c[Elt<ESZ>::EPC], s[Elt<ESZ>::EPC];
                        load_cs<ESZ>(P.cs + cs + pl.cs_off, un[w], c, s);
                        apply_rot<ESZ>(un[w], va[w], vb[w], c, s);
                    }
                    char* d = dst_page + int64_t(r) * pl.token_stride;
                    st16(d + int64_t(un[w].a) * 16, va[w]);
                    if (un[w].b >= 0) st16(d + int64_t(un[w].b) * 16, vb[w]);
                }
            }
        }
        return;
    }

    // REMAP: rotate the rotary bands of a re-used page in place.
    if (pl.rot_units == 0) return;
    const KRemapTask T = P.remap_tasks[task - P.n_asm];
    const KSeqEntry S = P.seqs[T.seq];
    const KDirEntry& D = P.dirs[T.dir];
    if (D.cs < 0) return;
    const int64_t lo = int64_t(T.k) * P.page_size;
    const int valid = int(min(int64_t(P.page_size), int64_t(S.new_len) - lo));
    const int32_t pg = P.bt_in[int64_t(T.seq) * P.bt_stride + T.src_page];
    if (pg < 0 || pg >= P.capacity) {
        if (P.status && threadIdx.x == 0) atomicOr(P.status, int(LEYLINE_STATUS_BAD_PAGE));
        return;
    }
    char* page = pl.base + lbase_off + int64_t(pg) * pl.page_stride;
    const int32_t RU = pl.rot_units;
    const int32_t total = valid * RU;
    for (int32_t f = threadIdx.x; f < total; f += TPB) {
        const int32_t r = f / RU;
        const Unit un = map_rot_unit<ESZ>(pl, f - r * RU);
        char* row = page + int64_t(r) * pl.token_stride;
        float c[Elt<ESZ>::EPC], s[Elt<ESZ>::EPC];
        load_cs<ESZ>(P.cs + D.cs + pl.cs_off, un, c, s);
        u32x4 va = ld16(row + int64_t(un.a) * 16), vb;
        if (un.b >= 0) vb = ld16(row + int64_t(un.b) * 16);
        apply_rot<ESZ>(un, va, vb, c, s);
        st16(row + int64_t(un.a) * 16, va);
        if (un.b >= 0) st16(row + int64_t(un.b) * 16, vb);
    }
}

// New block tables and the freed-page list, resolved from the symbolic plan.
__global__ __launch_bounds__(TPB) void paged_tables_kernel(const KTableParams P) {
    const int64_t i = int64_t(blockIdx.x) * TPB + threadIdx.x;
    if (i < P.n_pages) {
        const KPageEntry e = P.pages[i];
        const int64_t row = i / P.bt_stride;
        int32_t v = -1;
        if (e.kind == LEYLINE_PAGE_IDENTITY || e.kind == LEYLINE_PAGE_REMAP)
            v = P.bt_in[row * P.bt_stride + e.src];
        else if (e.kind == LEYLINE_PAGE_ASSEMBLE)
            v = e.src < P.n_free ? P.free_pages[e.src] : -1;
        P.bt_out[i] = v;
    } else if (i < int64_t(P.n_pages) + P.n_freed) {
        const KFreedEntry f = P.freed[i - P.n_pages];
        P.freed_out[i - P.n_pages] = P.bt_in[int64_t(f.seq) * P.bt_stride + f.page];
    }
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
int launch(K kernel, dim3 grid, hipStream_t stream, const A& args) {
    (void)hipGetLastError();
    hipLaunchKernelGGL(kernel, grid, dim3(TPB), 0, stream, args);
    return hip_status(hipGetLastError());
}

}  // namespace

}  // namespace leyline

using namespace leyline;

extern "C" const char* leyline_last_hip_error(void) {
    return hipGetErrorString(g_last_hip_error);
}

extern "C" int leyline_splice_contig(const leyline_cache* cache, int64_t seq_len,
                                     const leyline_directive* dirs, int32_t n_dirs,
                                     int64_t* new_len_out, void* stream) {
    ContigSchedule sched;
    int rc = plan_contig(cache, seq_len, dirs, n_dirs, &sched);
    if (rc) return rc;
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    rc = describe_cache(cache, false, planes, &n_planes);
    if (rc) return rc;
    // every (job, plane) item's thread count must fit a 32-bit index
    for (const auto& jobs : sched.launches)
        for (const auto& j : jobs)
            for (int p = 0; p < n_planes; ++p) {
                const int64_t rows = j.is_stub ? j.count : std::min<int64_t>(j.count, j.delta < 0 ? -j.delta : j.delta);
                if (rows * planes[p].units > INT32_MAX - TPB) return LEYLINE_E_INVAL;
            }
    hipStream_t s = static_cast<hipStream_t>(stream);
    for (const auto& jobs : sched.launches) {
        KContigParams P;
        std::memset(&P, 0, sizeof(P));
        std::memcpy(P.planes, planes, sizeof(planes));
        P.n_layers = cache->n_layers;
        std::vector<KCosSin> cs;
        int32_t blocks = 0;
        int n_items = 0;
        for (size_t ji = 0; ji < jobs.size(); ++ji) {
            const ContigJobHost& j = jobs[ji];
            KContigJob& k = P.jobs[ji];
            k.src0 = j.src0;
            k.dst0 = j.dst0;
            k.count = j.count;
            k.delta = j.delta;
            k.is_stub = j.is_stub ? 1 : 0;
            k.chains = int32_t(j.is_stub ? j.count : std::min<int64_t>(j.count, j.delta < 0 ? -j.delta : j.delta));
            k.cs = -1;
            if (!j.is_stub && cos_sin_per_shift(cache) > 0) k.cs = append_cos_sin(cache, j.delta, cs);
            if (j.is_stub)
                for (int p = 0; p < n_planes; ++p) k.stub[p] = static_cast<const char*>(dirs[j.dir].stub[p]);
            for (int p = 0; p < n_planes; ++p) {
                const int64_t threads = int64_t(k.chains) * planes[p].units;
                blocks += int32_t((threads + TPB - 1) / TPB);
                P.item_job[n_items] = int32_t(ji);
                P.item_plane[n_items] = p;
                P.item_block_end[n_items] = blocks;
                ++n_items;
            }
        }
        P.n_items = n_items;
        if (cs.size() > size_t(KMAX_CS)) return LEYLINE_E_INVAL;
        std::copy(cs.begin(), cs.end(), P.cs);
        if (blocks == 0) continue;
        const dim3 grid(unsigned(blocks), unsigned(cache->n_layers));
        rc = cache->dtype == LEYLINE_BF16 ? launch(contig_splice_kernel<2>, grid, s, P)
                                          : launch(contig_splice_kernel<4>, grid, s, P);
        if (rc) return rc;
    }
    if (new_len_out) *new_len_out = sched.new_len;
    return LEYLINE_OK;
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
    KRotateParams P;
    std::memset(&P, 0, sizeof(P));
    int32_t upr = 0;
    for (int p = 0; p < n_planes; ++p) upr += planes[p].rot_units;
    if (n_rows == 0 || upr == 0 || delta == 0) return LEYLINE_OK;   // R(0) is the identity
    std::memcpy(P.planes, planes, sizeof(planes));
    P.n_planes = n_planes;
    P.n_layers = cache->n_layers;
    P.page_size = paged ? cache->page_size : 0;
    P.total_rows = total_rows;
    P.rows = rows;
    P.row0 = row0;
    P.n_rows = n_rows;
    P.status = device_status;
    P.units_per_row = upr;
    std::vector<KCosSin> cs;
    append_cos_sin(cache, delta, cs);
    std::copy(cs.begin(), cs.end(), P.cs);
    const int64_t blocks = (n_rows * upr + TPB - 1) / TPB;
    if (blocks > INT32_MAX) return LEYLINE_E_INVAL;
    const dim3 grid(unsigned(blocks), unsigned(cache->n_layers));
    hipStream_t s = static_cast<hipStream_t>(stream);
    return cache->dtype == LEYLINE_BF16 ? launch(rotate_rows_kernel<2>, grid, s, P)
                                        : launch(rotate_rows_kernel<4>, grid, s, P);
}

extern "C" int leyline_splice_paged(const leyline_cache* cache, int32_t n_seqs, const int32_t* seq_lens,
                                    const int32_t* block_table_in, int32_t* block_table_out, int32_t bt_stride,
                                    const leyline_directive* dirs, int32_t n_dirs,
                                    const int32_t* free_pages, int32_t n_free,
                                    int32_t* freed_pages_out, int32_t freed_cap,
                                    int32_t* new_seq_lens_out, int32_t* n_fresh_used_out, int32_t* n_freed_out,
                                    int32_t* device_status,
                                    void* workspace, int64_t workspace_bytes, void* stream) {
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    int rc = describe_cache(cache, true, planes, &n_planes);
    if (rc) return rc;
    if (cache->page_size > MAX_PAGE || bt_stride < 1 || n_free < 0 || freed_cap < 0) return LEYLINE_E_INVAL;
    if (n_seqs > 0 && (!block_table_in || !block_table_out || block_table_in == block_table_out))
        return LEYLINE_E_INVAL;
    PagedPlan plan;
    rc = plan_paged(cache->page_size, n_seqs, seq_lens, dirs, n_dirs, n_planes, &plan);
    if (rc) return rc;
    rc = check_table_width(plan, seq_lens, bt_stride);
    if (rc) return rc;
    if (plan.n_fresh > n_free) return LEYLINE_E_CAPACITY;
    if (int64_t(plan.freed_page.size()) > freed_cap) return LEYLINE_E_CAPACITY;
    if (plan.n_fresh > 0 && !free_pages) return LEYLINE_E_INVAL;
    if (!plan.freed_page.empty() && !freed_pages_out) return LEYLINE_E_INVAL;
    PagedImage img;
    rc = build_paged_image(cache, plan, n_seqs, dirs, n_dirs, bt_stride, &img);
    if (rc) return rc;
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < img.tables.total)
        return LEYLINE_E_WORKSPACE;

    hipStream_t s = static_cast<hipStream_t>(stream);
    const KPagedTables& t = img.tables;
    char* ws = static_cast<char*>(workspace);
    if (t.total > 0) {
        rc = hip_status(hipMemcpyAsync(ws, img.bytes.data(), size_t(t.total), hipMemcpyHostToDevice, s));
        if (rc) return rc;
    }
    if (t.n_asm + t.n_remap > 0) {
        KPagedParams P;
        std::memset(&P, 0, sizeof(P));
        std::memcpy(P.planes, planes, sizeof(planes));
        P.n_planes = n_planes;
        P.n_layers = cache->n_layers;
        P.page_size = cache->page_size;
        P.bt_stride = bt_stride;
        P.n_asm = t.n_asm;
        P.n_remap = t.n_remap;
        P.capacity = cache->capacity;
        P.seqs = reinterpret_cast<const KSeqEntry*>(ws + t.off_seq);
        P.dirs = reinterpret_cast<const KDirEntry*>(ws + t.off_dir);
        P.cs = reinterpret_cast<const KCosSin*>(ws + t.off_cs);
        P.asm_tasks = reinterpret_cast<const KAssembleTask*>(ws + t.off_asm);
        P.remap_tasks = reinterpret_cast<const KRemapTask*>(ws + t.off_remap);
        P.bt_in = block_table_in;
        P.free_pages = free_pages;
        P.n_free = n_free;
        P.status = device_status;
        const dim3 grid(unsigned(t.n_asm + t.n_remap), unsigned(cache->n_layers), unsigned(n_planes));
        rc = cache->dtype == LEYLINE_BF16 ? launch(paged_splice_kernel<2>, grid, s, P)
                                          : launch(paged_splice_kernel<4>, grid, s, P);
        if (rc) return rc;
    }
    if (t.n_pages + t.n_freed > 0) {
        KTableParams T;
        std::memset(&T, 0, sizeof(T));
        T.pages = reinterpret_cast<const KPageEntry*>(ws + t.off_pages);
        T.freed = reinterpret_cast<const KFreedEntry*>(ws + t.off_freed);
        T.bt_in = block_table_in;
        T.bt_out = block_table_out;
        T.free_pages = free_pages;
        T.freed_out = freed_pages_out;
        T.status = device_status;
        T.capacity = cache->capacity;
        T.n_pages = t.n_pages;
        T.n_freed = t.n_freed;
        T.bt_stride = bt_stride;
        T.n_free = n_free;
        const int64_t blocks = (int64_t(t.n_pages) + t.n_freed + TPB - 1) / TPB;
        rc = launch(paged_tables_kernel, dim3(unsigned(blocks)), s, T);
        if (rc) return rc;
    }
    if (new_seq_lens_out)
        for (int32_t b = 0; b < n_seqs; ++b) new_seq_lens_out[b] = plan.new_lens[size_t(b)];
    if (n_fresh_used_out) *n_fresh_used_out = plan.n_fresh;
    if (n_freed_out) *n_freed_out = int32_t(plan.freed_page.size());
    return LEYLINE_OK;
}
