// Plain-old-data parameter blocks shared by the host planner (built with the host compiler)
// and the HIP kernels (built with hipcc).  Layouts must stay identical on both sides: only
// fixed-width integers, floats and raw pointers.
#pragma once

#include <climits>
#include <cstdint>

#include "leyline.h"

// Functions used by both the kernels and host-side checks of their schedules.
#if defined(__HIPCC__)
#define LEYLINE_HD __host__ __device__
#else
#define LEYLINE_HD
#endif

namespace leyline {

// Rows are moved as 16-byte vectors ("chunks").  In the row kernels one thread moves one chunk
// of a row, except for half-split (NEOX) bands whose halves cannot be exchanged between lanes of
// a wavefront (neox_lanes == 0): there a thread moves a low-half chunk and its partner (a
// "two-chunk unit").  Rotary-only kernels (rotate in place) map threads over the bands alone.
enum : int32_t { KROT_NONE = 0, KROT_INTERLEAVED = 1, KROT_NEOX = 2 };

// Division by a fixed divisor d: n / d == (umulhi(n, mul) + n) >> shift for 0 <= n < 2^31.
struct KDiv {
    uint32_t mul;
    int32_t shift;
};

struct KPlane {
    char* base;              // device
    int64_t layer_stride;    // bytes
    int64_t token_stride;    // bytes
    int64_t page_stride;     // bytes (paged caches)
    int32_t row_bytes;
    int32_t row_chunks;      // row_bytes / 16
    int32_t rot;             // KROT_*
    int32_t n_heads;
    int32_t head_chunks;     // head stride in chunks
    int32_t rot_lo;          // first rotary chunk within a head
    int32_t rot_chunks;      // rotary band length in chunks (whole band, both halves)
    int32_t cs_off;          // offset of this plane's pairs within one shift's cos/sin block
    int32_t n_pairs;         // rotary pairs per head (rot_dim / 2)
    int32_t neox_lanes;      // 1: half-split partners are exchanged between lanes of a wavefront
    int32_t neox_dpp;        // 1: ... and every band is 16 chunks on 16-chunk boundaries, so a
                             // lane's partner is lane ^ 8 within its row of 16 lanes (DPP)
    int32_t band_wide;       // 1: the rotary bands make up at least half of the row (GQA K),
                             // 0: a narrow slice of each row (MLA K_pe)
    int32_t tpr;             // row kernels: threads per row (row_chunks, or two-chunk units)
    int32_t units_all;       // two-chunk units per row (ordered-chain kernel)
    KDiv tpr_div;            // division by tpr
    KDiv head_div;           // division by head_chunks
    KDiv uhead_div;          // division by head_chunks - rot_chunks/2 (two-chunk units per head)
    int32_t band_tpr;        // rotary-only kernels: threads per band (rot_chunks, or half of it)
    int32_t rot_tpr;         // rotary-only kernels: threads per row (n_heads * band_tpr)
    KDiv band_div;           // division by band_tpr
    // Row kernels, narrow interleaved bands of one head: pack_groups = B > 0 lays the rows out in
    // blocks of B row groups whose band chunks (B * rot_chunks = 64) come first, as one wavefront,
    // and their other chunks after, so that only one wavefront in (B * tpr / 64) rotates.
    int32_t pack_groups;
    int32_t pack_nb_shift;   // log2(rot_chunks) when packing
    KDiv pack_div;           // division by pack_groups * tpr
    KDiv rest_div;           // division by tpr - rot_chunks
};

// Precision of the pair arithmetic.  0: fp32 cos/sin and fp32 products (the paper's policy);
// 1: fp64 cos/sin and fp64 products, each result rounded once to the storage dtype, which makes
// the stored values the correctly rounded ones of the exact rotation (up to fp64 rounding).
#ifndef LEYLINE_PAIR_F64
#define LEYLINE_PAIR_F64 0
#endif
// The gather kernel, and with fp64 pairs the round kernel too, lay the band chunks of narrow
// interleaved bands (MLA K_pe) out in wavefronts of their own, so that the other wavefronts carry
// no pair arithmetic (KPlane::pack_groups).  Round kernel, 32K MLA splice: fp64 pairs 74.3% ->
// 78.4% of peak, fp32 pairs 79.2% -> 78.8%, so the fp32 build keeps its rows end to end there;
// fp32 gathers gain 0.6-2.3 points.
#ifndef LEYLINE_ROUND_PACK
#define LEYLINE_ROUND_PACK LEYLINE_PAIR_F64
#endif
// The same in the ordered-tile kernel, whose packed items use tiles of whole packed blocks.
#ifndef LEYLINE_TILE_PACK
#define LEYLINE_TILE_PACK LEYLINE_PAIR_F64
#endif

#if LEYLINE_PAIR_F64
typedef double kcs_t;
#else
typedef float kcs_t;
#endif

struct KCosSin {
    kcs_t c, s;
};

// fp64 -> fp32 rounded to odd: the value truncated toward zero, with the last bit set when the
// conversion was inexact.  Rounding this float to nearest-even bf16 (16 bits fewer) gives the
// nearest-even bf16 of the fp64 value itself: rounding to odd with at least two extra bits and
// then to nearest is one correct rounding (Boldo and Melquiond, "Emulation of FMA and correctly
// rounded sums: proved algorithms using rounding to odd", 2008).  Built from the nearest-even
// conversion: an inexact result whose last bit is even is replaced by its neighbour on the side
// of the fp64 value, which is then the odd one of the two floats around it.
LEYLINE_HD inline float f32_round_odd(double d) {
    const float f = float(d);
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    if (double(f) != d && !(u & 1u)) u += __builtin_fabs(d) > __builtin_fabs(double(f)) ? 1u : 0xffffffffu;
    return __builtin_bit_cast(float, u);
}

// ------------------------------------------------------------------------------ contiguous --
constexpr int KMAX_JOBS = 6;
// cos/sin pairs one launch carries in its kernel arguments (and stages in LDS); sized so that the
// argument blocks stay within 3.4 KB whatever the pair precision
constexpr int KMAX_CS = LEYLINE_PAIR_F64 ? 120 : 192;



// Kinds of contiguous jobs.
enum : int32_t {
    KJOB_ROUND = 0,   // rows [src0, src0+count) move by delta with count <= |delta|: sources and
                      // destinations are disjoint, one chunk per thread
    KJOB_CHAIN = 1,   // rows [src0, src0+count) move by delta, count > |delta|: ordered chains
                      // (layouts whose half-split partners need two-chunk units)
    KJOB_STUB = 2,    // count replacement rows copied to [dst0, dst0+count)
    KJOB_TILE = 3     // rows [src0, src0+count) move by delta as ordered tiles
};

// One (job, plane) item of a round, chain or replacement launch, self-contained so that a
// workgroup reads its parameters with one level of independent scalar loads (blockIdx.z selects
// the item).
struct KItem {
    KPlane pl;
    const char* stub;        // KJOB_STUB: dense [layers][count][row] for this plane
    int64_t src0;            // move: first source row
    int64_t dst0;            // stub: first destination row
    int64_t count;           // rows
    int64_t delta;           // move: nonzero shift
    int32_t kind;            // KJOB_*
    int32_t chains;          // chain: min(|delta|, count)
    int32_t cs;              // first cos/sin entry of this plane's pairs (-1: no rotation)
    int32_t pad;
};

constexpr int KMAX_LAUNCH_ITEMS = 8;

struct KContigParams {
    KItem items[KMAX_LAUNCH_ITEMS];
    int32_t block0[KMAX_LAUNCH_ITEMS];   // round and replacement launches: first workgroup (x) of
                                         // each item, side by side; INT32_MAX past n_items
    int32_t n_items;
    int32_t n_layers;
    KCosSin cs[KMAX_CS];
};

// Ordered tiles: chunks per thread and per tile (one tile = one workgroup, one layer).
#ifndef LEYLINE_TILE_CPT
#define LEYLINE_TILE_CPT 8
#endif
#ifndef LEYLINE_TILE_TPB
#define LEYLINE_TILE_TPB 1024
#endif
constexpr int KTILE_CPT = LEYLINE_TILE_CPT;
constexpr int KTILE_TPB = LEYLINE_TILE_TPB;
constexpr int KTILE_CHUNKS = KTILE_TPB * KTILE_CPT;
// A call whose full-size tiles number fewer than KTILE_SMALL_TICKETS (over all layers) cannot
// fill the device and runs in tiles of KTILE_SMALL_CHUNKS chunks instead (the same kernel, which
// skips the load slots that no thread of a short tile needs).
#ifndef LEYLINE_TILE_SMALL_TICKETS
#define LEYLINE_TILE_SMALL_TICKETS 96
#endif
constexpr int KTILE_SMALL_TICKETS = LEYLINE_TILE_SMALL_TICKETS;
constexpr int KTILE_SMALL_CHUNKS = KTILE_CHUNKS / 4;

// One (job, plane) item of an ordered-tile launch: a move (rows [src0, src0 + count) to
// [dst0, dst0 + count), dst0 = src0 + delta) or a replacement copy (rows of `stub` to
// [dst0, dst0 + count)), cut into n_tiles tiles per layer.
struct KTileItem {
    int64_t src0;
    int64_t dst0;
    int64_t count;
    int64_t delta;           // move: nonzero shift; replacement: 0
    const char* stub;        // replacement: dense [layers][count][row] of this plane
    int32_t kind;            // KJOB_TILE (move) or KJOB_STUB
    int32_t plane;
    int32_t cs;              // first entry of the call's cos/sin table for this plane (-1: none)
    int32_t n_tiles;         // tiles per layer
    int32_t ticket0;         // first ticket of the item in its launch
    int32_t flag0;           // move: first "source read" flag, one per (layer, tile in
                             // processing order) at layer * n_tiles + tile; replacement: -1
    uint32_t waits;          // bit a: item a of the launch, an earlier move of the same plane,
                             // reads rows this item writes
    int32_t tile_chunks;     // chunks per tile: KTILE_CHUNKS, or a whole number of packed blocks
    int32_t pack;            // 1: units laid out by row_unit with packed bands (tiles of whole rows)
    int32_t pad;
};

constexpr int KTILE_MAX_ITEMS = 24;

// A tile's wait for one flag gives up after this many unsuccessful polls, each followed by a
// short sleep (at least a few hundred milliseconds in all).  In a correct schedule the awaited
// tile has already taken its ticket and only has its own loads to finish, which takes
// microseconds; the bound turns a schedule fault (or a workspace shared by calls that overlap)
// into a status bit and skipped stores instead of a workgroup that never exits.
constexpr int32_t KTILE_SPIN_LIMIT = 1 << 22;

// Polls ready() until it returns true, with pause() between polls, at most `limit` failed polls:
// whether the wait succeeded.  The tile kernel waits this way; the CPU schedule simulator models
// its give-up path with it.
template <class R, class S>
LEYLINE_HD inline bool tile_wait_bounded(R&& ready, S&& pause, int32_t limit) {
    for (int32_t i = 0; i < limit; ++i) {
        if (ready()) return true;
        pause();
    }
    return ready();
}

struct KTileParams {
    KPlane planes[LEYLINE_MAX_PLANES];
    KTileItem items[KTILE_MAX_ITEMS];
    int32_t ticket0[KTILE_MAX_ITEMS];   // items[i].ticket0, side by side; INT32_MAX past n_items
    int32_t n_items;
    int32_t n_tickets;
    int32_t* counter;        // ticket counter of this launch, zero before it
    int32_t* flags;          // the call's flags, zero before the first tile launch
    const KCosSin* cs;       // the call's cos/sin table
    int32_t* status;         // device, nullable: LEYLINE_STATUS_TILE_TIMEOUT on a wait given up
};

// The side-by-side table of the items' first tickets (INT32_MAX past the last item), filled by
// the host before a tile launch.
inline void tile_fill_ticket_table(KTileParams& P) {
    for (int32_t i = 0; i < KTILE_MAX_ITEMS; ++i) P.ticket0[i] = i < P.n_items ? P.items[i].ticket0 : INT32_MAX;
}

// The item of a tile launch that owns `ticket`: items hold ascending ticket ranges, so its index
// is the number of later items whose range starts at or before the ticket (a fixed number of
// independent reads, no loop-carried dependency).
LEYLINE_HD inline int32_t tile_item_of(const KTileParams& P, int32_t ticket) {
    int32_t it = 0;
    for (int32_t i = 1; i < KTILE_MAX_ITEMS; ++i) it += ticket >= P.ticket0[i] ? 1 : 0;
    return it;
}

LEYLINE_HD inline int64_t kmin64(int64_t a, int64_t b) { return a < b ? a : b; }
LEYLINE_HD inline int64_t kmax64(int64_t a, int64_t b) { return a > b ? a : b; }

// The flags that tile `order` (processing order) of item `it` of a tile launch, in `layer`, waits
// for before it stores: f(i) for the flag word i of the call's flags, once per overlapping tile
// (possibly for one flag more than once).  A move's tile waits for the earlier tiles of its own
// move whose source its destination overlaps: the shift is M chunks, so the tiles floor(M/C) and
// ceil(M/C) places earlier in processing order.  Any tile then waits for the tiles of the earlier
// moves listed in its item's `waits` whose source rows overlap its destination rows.
template <class F>
LEYLINE_HD inline void tile_wait_flags(const KTileParams& P, int32_t it, int32_t layer, int32_t order, F&& f) {
    const KTileItem& I = P.items[it];
    const int64_t tpr = P.planes[I.plane].tpr;
    const bool down = I.delta <= 0;
    const int64_t q = down ? order : I.n_tiles - 1 - order;
    if (I.kind == KJOB_TILE) {
        const int64_t M = (down ? -I.delta : I.delta) * tpr;
        const int64_t T = I.tile_chunks;
        for (int64_t d = M / T; d <= (M + T - 1) / T; ++d) {
            const int64_t j = order - d;
            if (d == 0 || j < 0) continue;
            f(I.flag0 + int64_t(layer) * I.n_tiles + j);
        }
    }
    uint32_t w = I.waits;
    if (!w) return;
    const int64_t c_hi = kmin64((q + 1) * I.tile_chunks, I.count * tpr);
    const int64_t lo = I.dst0 + q * I.tile_chunks / tpr;                // destination rows [lo, hi)
    const int64_t hi = I.dst0 + (c_hi - 1) / tpr + 1;
    while (w) {
        const int a = __builtin_ctz(w);
        w &= w - 1;
        const KTileItem& A = P.items[a];
        const int64_t x0 = kmax64(lo, A.src0), x1 = kmin64(hi, A.src0 + A.count);
        if (x0 >= x1) continue;
        const int64_t t0 = (x0 - A.src0) * tpr / A.tile_chunks;
        const int64_t t1 = ((x1 - A.src0) * tpr - 1) / A.tile_chunks;
        for (int64_t t = t0; t <= t1; ++t) {
            const int64_t o = A.delta < 0 ? t : A.n_tiles - 1 - t;     // A's processing order
            f(A.flag0 + int64_t(layer) * A.n_tiles + o);
        }
    }
}

// Before the tile launches of a call: clear its counters and flags, and write entries of its
// cos/sin table into the workspace (carried here, in the kernel arguments).
constexpr int KPREP_CS = LEYLINE_PAIR_F64 ? 208 : 320;

struct KPrepParams {
    int32_t* zero;
    int64_t n_zero;          // 32-bit words from `zero`
    KCosSin* cs_dst;
    int32_t n_cs;            // entries of cs[] written to cs_dst
    int32_t pad;
    KCosSin cs[KPREP_CS];
};

// ------------------------------------------------------------------------------ rotate-only --
// The rotation's scalars, side by side so that a workgroup reads them as one value.
struct KRotateHead {
    int32_t n_planes;
    int32_t n_layers;
    int32_t page_size;       // 0: contiguous
    int32_t pad;
    int64_t total_rows;      // bound for listed rows
    const int64_t* rows;     // device, nullable
    int64_t row0;
    int64_t n_rows;
    int32_t* status;         // device, nullable
};

struct KRotateParams {
    KPlane planes[LEYLINE_MAX_PLANES];
    KRotateHead h;
    KDiv rot_div[LEYLINE_MAX_PLANES];   // by rot_tpr (band units per row)
    KDiv page_div;           // by page_size (paged caches)
    int32_t rot_base[LEYLINE_MAX_PLANES + 1];   // workgroups of plane p: [rot_base[p], rot_base[p+1])
    int32_t pad3;
    KCosSin cs[KMAX_CS];
};

// ----------------------------------------------------------------------------------- paged --
struct KSeqEntry {
    int32_t dir_begin, dir_count;   // the sequence's directives
    int32_t new_len;
    int32_t run_begin, run_count;   // the sequence's page runs
    int32_t pad0, pad1, pad2;
};

struct KDirEntry {
    int64_t stub_start;      // new position of the replacement's first token
    int64_t stub_len;
    int64_t delta;           // cumulative shift of the segment that follows the replacement
    int32_t cs;              // first cos/sin entry of that shift (-1: shift 0 or no rotary plane)
    int32_t pad;
    const char* stub[LEYLINE_MAX_PLANES];
};

// A run of consecutive new logical pages [k0, k0 + count) of one sequence that share a kind.
// IDENTITY and REMAP: page k0 + c re-uses old logical page src0 + c; ASSEMBLE: it takes fresh
// ordinal src0 + c.  ord0 is the ordinal of the run's first page among all pages of its kind in
// the call (ASSEMBLE: equal to src0); dir is the directive whose shift a REMAP run applies.
struct KPageRun {
    int32_t seq, k0, count, kind, src0, ord0, dir, pad;
};

// Old logical pages [page0, page0 + count) of one sequence that the call drops, written to
// freed-list positions [out0, out0 + count).
struct KFreedRun {
    int32_t seq, page0, count, out0;
};

// One row of an ASSEMBLE page, resolved on the device from the plan and the block tables.
struct KRowMove {
    int32_t src_page;        // physical page of the old row; KROW_STUB: replacement row; KROW_SKIP
    int32_t src_row;         // row within that page, or token of the replacement
    int32_t dst_page;        // fresh physical page
    int32_t dst_row;         // row within the fresh page
    int32_t cs;              // first cos/sin entry of the row's shift (-1: not rotated)
    int32_t dir;             // replacement rows: directive index
};
constexpr int32_t KROW_STUB = -1;
constexpr int32_t KROW_SKIP = -2;

// One REMAP page, resolved on the device by the workgroups that rotate it: its physical page, the
// cos/sin entry of its shift and the number of valid rows (0: nothing to rotate).
struct KRemapPage {
    int32_t page, cs, rows, pad;
};

// Byte offsets of the tables inside the workspace (converted to pointers at launch).
struct KPagedTables {
    int64_t off_seq, off_dir, off_cs, off_runs, off_asm_runs, off_remap_runs, off_freed_runs;
    int64_t off_rows, off_order, off_remap_sorted;
    int64_t upload;          // bytes uploaded from the host (the tables before the row tables)
    int64_t total;           // workspace bytes (the row table is written on the device)
    int32_t n_seqs, n_dirs, n_cs, n_runs, n_asm_runs, n_remap_runs, n_freed_runs;
    int32_t n_asm, n_remap, n_freed, bt_stride;
    int32_t n_rows;          // n_asm * page_size
    int32_t remap_sorted;    // 1: the REMAP pages are laid out in physical order at off_remap_sorted
};

// Plans of at most this many bytes travel in the kernel arguments instead of being uploaded.
constexpr int32_t KPLAN_INLINE = 2560;

struct KPagedParams {
    KPlane planes[LEYLINE_MAX_PLANES];
    int32_t n_planes;
    int32_t n_layers;
    int32_t page_size;
    int32_t bt_stride;
    int32_t n_asm;
    int32_t n_remap;
    int32_t n_rows;          // ASSEMBLE rows (n_asm * page_size)
    int32_t order_shift;     // destination-order bucket = physical page >> order_shift
    KDiv remap_div[LEYLINE_MAX_PLANES];  // by page_size * rot_tpr (band units per REMAP page)
    KDiv rot_div[LEYLINE_MAX_PLANES];    // by rot_tpr (band units per row)
    int64_t capacity;                    // physical pages
    // plan tables: at `plan` (the workspace copy), or, when plan is null, in `blob` below (a plan
    // small enough to travel in the kernel arguments); byte offsets within either
    const char* plan;
    int32_t off_seq, off_dir, off_cs, off_runs, off_asm_runs, off_remap_runs, off_freed_runs;
    int32_t n_asm_runs, n_remap_runs;
    const int32_t* bt_in;
    const int32_t* free_pages;
    int32_t n_free;
    int32_t table_blocks;    // data kernel: workgroups writing the block tables and the freed list
                             // (0: the resolve kernel writes them)
    int32_t layer_groups;    // data kernel: groups of PAGED_LPT layers
    KDiv move_blk_div;       // data kernel: division by the gather workgroups of one layer group
    KDiv remap_blk_div;      // data kernel: division by the REMAP workgroups of one layer group
    int32_t* status;
    KRowMove* rows;          // workspace, n_rows entries (null: the gather resolves rows itself)
    // block tables and freed list
    int32_t* bt_out;
    int32_t* freed_out;
    int32_t n_table;         // n_seqs * bt_stride
    int32_t n_freed;
    int32_t n_freed_runs;
    int32_t move_base[LEYLINE_MAX_PLANES + 1];   // data kernel: gather workgroups of plane p are
                                                 // [move_base[p], move_base[p+1])
    int32_t remap_base[LEYLINE_MAX_PLANES + 1];  // then REMAP workgroups of plane p, numbered
                                                 // from 0 after the gather's
    int32_t gather_split;    // data kernel: 1 = each XCD gathers its own eighth (see xcd_eighth)
    int32_t* order;          // workspace, n_asm fresh ordinals in destination-page order (or null)
    KRemapPage* remap_sorted;   // workspace, the REMAP pages resolved and in physical-page order
                                // (or null: the rotating workgroups resolve them in plan order)
    int32_t remap_shift;     // its bucket = physical page >> remap_shift
    int32_t remap_pack;      // 1: a resolved REMAP page's shift index + 1 and rows fit 16 bits each
    // the only REMAP run when n_remap_runs == 1, with its shift's cos/sin entry and its sequence's
    // new length (read with the other parameters, one level of loads before the block table)
    KPageRun remap0;
    int32_t remap0_cs, remap0_len;
    alignas(16) unsigned char blob[KPLAN_INLINE];
};

// A call assembling at most this many rows gathers them without a row table: each gathering
// workgroup resolves its rows from the plan, and the whole call is one data launch.
constexpr int32_t KINLINE_ROWS = 1024;

// The gather is ordered by destination page (neighbouring physical pages processed together)
// when a call assembles at least this many pages; KORDER_BUCKETS buckets of pages, counted in LDS.
constexpr int32_t KORDER_MIN = 64;
constexpr int32_t KORDER_BUCKETS = 4096;

// The REMAP rotation runs in physical-page order (resolved and bucket-sorted by a first kernel)
// when a call re-uses at least KORDER_MIN pages and some plane rotates at least this many bytes
// per row (whole GQA K heads: neighbouring rows then share DRAM pages; narrow MLA bands gain
// nothing from it).
constexpr int32_t KREMAP_SORT_BYTES = 1024;


// n / d for 0 <= n < 2^31 with a KDiv (the kernels' multiply-shift division), on either side.
LEYLINE_HD inline int32_t kdiv(int32_t n, KDiv d) {
    const uint32_t hi = uint32_t((uint64_t(uint32_t(n)) * d.mul) >> 32);
    return int32_t((hi + uint32_t(n)) >> d.shift);
}

// Unit t of a row kernel's item (row groups of a few rows laid end to end, one chunk per unit):
// its row group g and chunk u (u < tpr for every t, also past the item's last group).  With pack
// and pack_groups = B, units come in blocks of B row groups: first the band chunks of the block's
// groups (rot_chunks each), then each group's other chunks in order.
LEYLINE_HD inline void row_unit(const KPlane& pl, bool pack, int32_t t, int64_t groups, int32_t& g, int32_t& u) {
    if (pack && pl.pack_groups) {
        const int32_t B = pl.pack_groups, nb = pl.rot_chunks;
        const int32_t blk = kdiv(t, pl.pack_div);
        const int32_t w = t - blk * B * pl.tpr;
        const int32_t g0 = blk * B;
        const int64_t left = groups - int64_t(g0);
        const int32_t gb = int32_t(left <= 0 ? 0 : left < B ? left : B);   // groups of this block
        if (w < gb * nb) {
            g = g0 + (w >> pl.pack_nb_shift);
            u = pl.rot_lo + (w & (nb - 1));
        } else {
            const int32_t w2 = w - gb * nb;
            const int32_t gi = kdiv(w2, pl.rest_div);
            const int32_t c = w2 - gi * (pl.tpr - nb);
            g = g0 + gi;
            u = c < pl.rot_lo ? c : c + nb;
        }
    } else {
        g = kdiv(t, pl.tpr_div);
        u = t - g * pl.tpr;
    }
}

}  // namespace leyline
