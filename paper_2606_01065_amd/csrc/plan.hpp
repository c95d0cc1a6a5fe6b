// Host-side planning for the splice kernels: validation of the C-ABI arguments, the order in
// which overlapping contiguous moves may run, paged page plans, and the fp64 -> fp32 cos/sin
// tables.  Pure C++ (no HIP calls) so that every rule here can be exercised without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "leyline.h"
#include "kparams.hpp"

namespace leyline {

// Multiply-shift constants for division by d (1 <= d < 2^31), exact for numerators < 2^31.
KDiv make_div(int32_t d);

// A validated plane, reduced to what the kernels need (byte strides, 16-byte chunk geometry).
int describe_cache(const leyline_cache* cache, bool paged, KPlane out[LEYLINE_MAX_PLANES],
                   int* n_planes);

// Validation of one sequence's directives (already restricted to that sequence, FORGET already
// resolved).
int check_sequence(int64_t seq_len, const leyline_directive* dirs, int32_t n_dirs,
                   int32_t n_planes);

// FORGET hands an edit to a prefix-trimmed re-prefill: on the cache it is the deletion of
// [span_start, seq_len) with no replacement.  Checks the FORGET rules (last directive of its
// sequence, no replacement, span inside the sequence) and, when a FORGET directive is present,
// copies the directives into *buf with each FORGET replaced by that deletion; *use points at the
// directives to plan with.  seq_lens: per sequence (paged), or NULL with seq_len (contiguous).
int resolve_forget(const leyline_directive* dirs, int32_t n_dirs, int32_t n_seqs,
                   const int32_t* seq_lens, int64_t seq_len, std::vector<leyline_directive>* buf,
                   const leyline_directive** use);

// cos/sin of (shift * theta_i), evaluated in fp64 and rounded to fp32, for every rotary pair of
// every rotary plane, appended to `table`.  Returns the offset of the first entry.
int32_t append_cos_sin(const leyline_cache* cache, int64_t shift, std::vector<KCosSin>& table);

// Number of cos/sin entries one shift needs (sum over rotary planes of rot_dim / 2).
int32_t cos_sin_per_shift(const leyline_cache* cache);

// ------------------------------------------------------------------------------------------
// Contiguous splice: a set of jobs (move a source range by a shift, or copy a stub) grouped
// into launches so that no job of a launch overwrites a row another job of the same or a later
// launch still has to read.
struct ContigJobHost {
    int32_t kind;       // KJOB_*
    int64_t src0, dst0, count, delta;
    int32_t dir;        // stub: directive index
};

// A move needing more rounds than this runs as ordered chains (or tiles) instead.
constexpr int64_t MAX_ROUNDS = 16;
// Rounds moving fewer bytes than this (all layers and planes) are not worth a launch each.
constexpr int64_t ROUND_MIN_BYTES = int64_t(64) << 20;

// One ordered-tile launch: its items (in dependency order) and its number of tickets.
struct TileLaunchHost {
    std::vector<KTileItem> items;
    int64_t tickets = 0;
};

struct ContigSchedule {
    int64_t new_len = 0;
    // Rounds, chains and replacement copies: groups of independent jobs, in order.
    std::vector<std::vector<ContigJobHost>> launches;
    // Ordered tiles (used for every job of a call once any move needs them): launches in order,
    // after prep launches that clear the workspace and write the cos/sin table into it.
    bool tiles = false;
    std::vector<TileLaunchHost> tile_launches;
    std::vector<KCosSin> cs;    // the call's cos/sin table (tiles)
    int64_t ws_flags = 0;       // workspace byte offsets: ticket counters (256 bytes per tile
    int64_t ws_cs = 0;          // launch) from 0, flags from ws_flags, cos/sin table from ws_cs
    int64_t ws_bytes = 0;       // workspace bytes (0 without tiles)
};

// Tiles of one ordered-tile move on a plane with `tpr` chunks per row.
int64_t tile_count(int64_t rows, int32_t tpr, int32_t tile_chunks);

int plan_contig(const leyline_cache* cache, int64_t seq_len, const leyline_directive* dirs,
                int32_t n_dirs, ContigSchedule* out);

// ------------------------------------------------------------------------------------------
// Paged splice.
// The plan is kept as runs of pages: its size grows with the number of directives and sequences,
// not with the number of pages.
struct PagedPlan {
    int32_t page_size = 0;
    int32_t n_seqs = 0;
    std::vector<leyline_directive> resolved;   // the directives with FORGET resolved (if any)
    const leyline_directive* dirs = nullptr;   // the directives the plan was made from
    std::vector<int32_t> new_lens;
    std::vector<int32_t> run_begin;    // [n_seqs + 1]: sequence b owns runs [run_begin[b], run_begin[b+1])
    std::vector<KPageRun> runs;        // ascending (seq, k0); they cover every new page exactly once
    std::vector<KFreedRun> freed;      // ascending (seq, page0)
    int32_t n_fresh = 0;               // ASSEMBLE pages (fresh pages consumed)
    int32_t n_remap = 0;
    int32_t n_freed = 0;
};

// remap = false: copy-on-write (no page whose rows shift is re-used; such pages are assembled).
int plan_paged(int32_t page_size, int32_t n_seqs, const int32_t* seq_lens,
               const leyline_directive* dirs, int32_t n_dirs, int32_t n_planes, bool remap,
               PagedPlan* out);

// E_CAPACITY unless every sequence's old and new page count fits a block-table row.
int check_table_width(const PagedPlan& plan, const int32_t* seq_lens, int32_t bt_stride);

// Device-side image of a paged plan (built into the caller's workspace).
struct PagedImage {
    std::vector<unsigned char> bytes;   // contents to upload
    KPagedTables tables;                // offsets into the workspace (pointers filled at launch)
};

int build_paged_image(const leyline_cache* cache, const PagedPlan& plan, int32_t n_seqs,
                      const leyline_directive* dirs, int32_t n_dirs, int32_t bt_stride,
                      PagedImage* img);

}  // namespace leyline
