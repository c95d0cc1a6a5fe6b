// Host planner of the splice library: argument validation, ordering of overlapping in-place
// moves, paged page plans and fp64 cos/sin tables.  No HIP calls: everything here runs and is
// tested without a GPU.
#include "plan.hpp"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <map>

namespace leyline {

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int elem_size(int32_t dtype) {
    if (dtype == LEYLINE_BF16) return 2;
    if (dtype == LEYLINE_F32) return 4;
    return 0;
}

}  // namespace

KDiv make_div(int32_t d) {
    int32_t l = 0;
    while ((int64_t(1) << l) < d) ++l;
    const uint64_t mul = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - uint64_t(d))) / uint64_t(d) + 1;
    return KDiv{uint32_t(mul), l};
}

int describe_cache(const leyline_cache* cache, bool paged, KPlane out[LEYLINE_MAX_PLANES],
                   int* n_planes) {
    if (!cache) return LEYLINE_E_INVAL;
    const int esz = elem_size(cache->dtype);
    if (!esz || cache->n_layers < 1 || cache->n_layers > 65535 || cache->n_planes < 1 ||
        cache->n_planes > LEYLINE_MAX_PLANES)
        return LEYLINE_E_INVAL;
    if (paged ? cache->page_size < 1 : cache->page_size != 0) return LEYLINE_E_INVAL;
    if (cache->capacity < 0) return LEYLINE_E_INVAL;
    int32_t cs_off = 0;
    for (int p = 0; p < cache->n_planes; ++p) {
        const leyline_plane& pl = cache->planes[p];
        KPlane& k = out[p];
        std::memset(&k, 0, sizeof(k));
        if (!pl.base || !aligned16(pl.base) || pl.row_elems <= 0) return LEYLINE_E_INVAL;
        const int64_t row_bytes = int64_t(pl.row_elems) * esz;
        if (row_bytes % 16) return LEYLINE_E_INVAL;
        if (pl.token_stride < pl.row_elems || pl.layer_stride < 0) return LEYLINE_E_INVAL;
        if ((pl.token_stride * esz) % 16 || (pl.layer_stride * esz) % 16) return LEYLINE_E_INVAL;
        if (cache->n_layers > 1 && pl.layer_stride == 0) return LEYLINE_E_INVAL;
        if (paged) {
            if (pl.page_stride < int64_t(cache->page_size) * pl.token_stride && cache->capacity > 1)
                return LEYLINE_E_INVAL;
            if ((pl.page_stride * esz) % 16) return LEYLINE_E_INVAL;
        }
        k.base = static_cast<char*>(pl.base);
        k.layer_stride = pl.layer_stride * esz;
        k.token_stride = pl.token_stride * esz;
        k.page_stride = paged ? pl.page_stride * esz : 0;
        k.row_bytes = int32_t(row_bytes);
        k.row_chunks = int32_t(row_bytes / 16);
        k.rot = KROT_NONE;
        k.tpr = k.row_chunks;
        k.head_chunks = k.row_chunks;
        if (pl.rot_dim != 0) {
            if (pl.rot_dim < 0 || (pl.rot_dim & 1) || pl.n_heads < 1 || pl.head_stride <= 0 ||
                pl.rot_offset < 0 || pl.rot_offset + pl.rot_dim > pl.head_stride ||
                int64_t(pl.n_heads) * pl.head_stride > pl.row_elems)
                return LEYLINE_E_INVAL;
            if (pl.rope_style != LEYLINE_ROPE_INTERLEAVED && pl.rope_style != LEYLINE_ROPE_NEOX)
                return LEYLINE_E_INVAL;
            if (!pl.inv_freq && !(pl.rope_base > 0.0)) return LEYLINE_E_INVAL;
            const bool neox = pl.rope_style == LEYLINE_ROPE_NEOX;
            if ((int64_t(pl.head_stride) * esz) % 16 || (int64_t(pl.rot_offset) * esz) % 16)
                return LEYLINE_E_INVAL;
            if ((int64_t(neox ? pl.rot_dim / 2 : pl.rot_dim) * esz) % 16) return LEYLINE_E_INVAL;
            k.rot = neox ? KROT_NEOX : KROT_INTERLEAVED;
            k.n_heads = pl.n_heads;
            k.head_chunks = int32_t(int64_t(pl.head_stride) * esz / 16);
            k.rot_lo = int32_t(int64_t(pl.rot_offset) * esz / 16);
            k.rot_chunks = int32_t(int64_t(pl.rot_dim) * esz / 16);
            k.n_pairs = pl.rot_dim / 2;
            k.cs_off = cs_off;
            cs_off += pl.rot_dim / 2;
            if (neox) {
                // Lane exchange in the row kernels: a wavefront covers 64 consecutive chunks of
                // the rows laid end to end, so every band must sit inside one 64-chunk window.
                bool ok = false;
                if (k.row_chunks % 64 == 0) {
                    ok = true;
                    for (int h = 0; h < k.n_heads; ++h) {
                        const int32_t lo = h * k.head_chunks + k.rot_lo, hi = lo + k.rot_chunks - 1;
                        if (lo / 64 != hi / 64) ok = false;
                    }
                } else if (64 % k.row_chunks == 0) {
                    ok = true;
                }
                k.neox_lanes = ok ? 1 : 0;
                if (!ok) k.tpr = k.row_chunks - k.n_heads * (k.rot_chunks / 2);
                // every kernel lays a lane's chunk at lane mod 16 of its 16-chunk group when rows
                // (row kernels) or bands (rotary-only kernels) are multiples of 16 chunks
                k.neox_dpp = (ok && k.rot_chunks == 16 && k.head_chunks % 16 == 0 && k.rot_lo % 16 == 0 &&
                              k.tpr % 16 == 0) ? 1 : 0;
            }
            k.band_wide = (2 * k.n_heads * k.rot_chunks >= k.row_chunks) ? 1 : 0;
            // rotary-only kernels pack the bands of consecutive heads and rows back to back
            k.band_tpr = (neox && !(k.rot_chunks <= 64 && !(k.rot_chunks & (k.rot_chunks - 1))))
                             ? k.rot_chunks / 2 : k.rot_chunks;
            k.rot_tpr = k.n_heads * k.band_tpr;
            // band chunks of 64 / rot_chunks row groups make one wavefront, the rest whole ones
            const int32_t nb = k.rot_chunks;
            if (k.rot == KROT_INTERLEAVED && k.n_heads == 1 && !k.band_wide && nb >= 1 && nb <= 64 &&
                (nb & (nb - 1)) == 0 && k.tpr == k.row_chunks && k.rot_lo + nb <= k.row_chunks &&
                (int64_t(64 / nb) * k.tpr) % 64 == 0) {
                k.pack_groups = 64 / nb;
                while ((1 << k.pack_nb_shift) < nb) ++k.pack_nb_shift;
                k.pack_div = make_div(k.pack_groups * k.tpr);
                k.rest_div = make_div(k.tpr - nb);
            }
        }
        k.units_all = k.rot == KROT_NEOX ? k.row_chunks - k.n_heads * (k.rot_chunks / 2) : k.row_chunks;
        k.tpr_div = make_div(k.tpr);
        k.head_div = make_div(k.head_chunks);
        k.uhead_div = make_div(std::max(1, k.head_chunks - k.rot_chunks / 2));
        k.band_div = make_div(std::max(1, k.band_tpr));
    }
    if (cs_off > KMAX_CS) return LEYLINE_E_INVAL;
    *n_planes = cache->n_planes;
    return LEYLINE_OK;
}

int32_t cos_sin_per_shift(const leyline_cache* cache) {
    int32_t n = 0;
    for (int p = 0; p < cache->n_planes; ++p) n += cache->planes[p].rot_dim / 2;
    return n;
}

int32_t append_cos_sin(const leyline_cache* cache, int64_t shift, std::vector<KCosSin>& table) {
    const int32_t first = int32_t(table.size());
    const double d = double(shift);   // exact: |shift| < 2^53
    for (int p = 0; p < cache->n_planes; ++p) {
        const leyline_plane& pl = cache->planes[p];
        const int half = pl.rot_dim / 2;
        for (int i = 0; i < half; ++i) {
            // theta_i = base^(-2i/d_rot) (RoFormer), or the caller's table
            const double theta = pl.inv_freq ? pl.inv_freq[i]
                                             : std::pow(pl.rope_base, -2.0 * i / pl.rot_dim);
            const double phi = d * theta;
            table.push_back(KCosSin{kcs_t(std::cos(phi)), kcs_t(std::sin(phi))});
        }
    }
    return first;
}

int check_sequence(int64_t seq_len, const leyline_directive* dirs, int32_t n_dirs,
                   int32_t n_planes) {
    if (n_dirs < 0 || (n_dirs > 0 && !dirs) || seq_len < 0) return LEYLINE_E_INVAL;
    int64_t prev_start = 0, prev_end = 0;
    for (int32_t j = 0; j < n_dirs; ++j) {
        const leyline_directive& d = dirs[j];
        if (d.mode != LEYLINE_AMORTIZE) return LEYLINE_E_INVAL;
        if (d.span_start < 0 || d.span_start > d.span_end || d.span_end > seq_len || d.stub_len < 0)
            return LEYLINE_E_RANGE;
        if (j > 0 && d.span_start < prev_start) return LEYLINE_E_ORDER;
        if (j > 0 && d.span_start < prev_end) return LEYLINE_E_OVERLAP;
        if (d.stub_len > 0)
            for (int p = 0; p < n_planes; ++p)
                if (!d.stub[p] || !aligned16(d.stub[p])) return LEYLINE_E_INVAL;
        prev_start = d.span_start;
        prev_end = d.span_end;
    }
    return LEYLINE_OK;
}

int resolve_forget(const leyline_directive* dirs, int32_t n_dirs, int32_t n_seqs,
                   const int32_t* seq_lens, int64_t seq_len, std::vector<leyline_directive>* buf,
                   const leyline_directive** use) {
    *use = dirs;
    if (n_dirs <= 0 || !dirs) return LEYLINE_OK;
    bool any = false;
    for (int32_t j = 0; j < n_dirs; ++j) {
        const leyline_directive& d = dirs[j];
        if (d.mode == LEYLINE_AMORTIZE) continue;
        if (d.mode != LEYLINE_FORGET) return LEYLINE_E_INVAL;
        if (j + 1 < n_dirs && dirs[j + 1].seq == d.seq) return LEYLINE_E_MODE;   // not the last
        if (d.stub_len != 0) return LEYLINE_E_MODE;
        if (seq_lens && (d.seq < 0 || d.seq >= n_seqs)) return LEYLINE_E_RANGE;
        const int64_t n = seq_lens ? seq_lens[d.seq] : seq_len;
        if (d.span_start < 0 || d.span_start > d.span_end || d.span_end > n) return LEYLINE_E_RANGE;
        any = true;
    }
    if (!any) return LEYLINE_OK;
    buf->assign(dirs, dirs + n_dirs);
    for (leyline_directive& d : *buf) {
        if (d.mode != LEYLINE_FORGET) continue;
        d.span_end = seq_lens ? seq_lens[d.seq] : seq_len;
        d.mode = LEYLINE_AMORTIZE;
    }
    *use = buf->data();
    return LEYLINE_OK;
}

// ------------------------------------------------------------------------------ contiguous --

int64_t tile_count(int64_t rows, int32_t tpr, int32_t tile_chunks) {
    return (rows * tpr + tile_chunks - 1) / tile_chunks;
}

namespace {

int64_t align256(int64_t v) { return (v + 255) & ~int64_t(255); }

// Every job of the call as ordered-tile items, in dependency-level order, packed into launches of
// at most KTILE_MAX_ITEMS items.  An item waits (inside its launch) for the earlier moves of its
// plane whose source rows it overwrites; items of earlier launches are finished by stream order.
// One cos/sin block per distinct shift goes into the call's table.  Tiles hold tile_base chunks
// (or a whole number of packed blocks up to that).
int plan_tiles(const leyline_cache* cache, const leyline_directive* dirs, const KPlane* planes,
               int n_planes, const std::vector<ContigJobHost>& jobs, const std::vector<int>& level,
               int32_t tile_base, ContigSchedule* out) {
    std::vector<size_t> order(jobs.size());
    for (size_t k = 0; k < order.size(); ++k) order[k] = k;
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return level[a] < level[b]; });
    const bool any_rot = cos_sin_per_shift(cache) > 0;
    std::map<int64_t, int32_t> shift_cs;                     // shift -> first entry of its block
    int64_t n_flags = 0;
    TileLaunchHost cur;
    out->tiles = true;
    for (size_t k : order) {
        const ContigJobHost& x = jobs[k];
        const bool move = x.kind != KJOB_STUB;
        if (int(cur.items.size()) + n_planes > KTILE_MAX_ITEMS) {
            out->tile_launches.push_back(std::move(cur));
            cur = TileLaunchHost();
        }
        int32_t cs0 = -1;
        if (move && any_rot) {
            const auto found = shift_cs.find(x.delta);
            if (found != shift_cs.end()) {
                cs0 = found->second;
            } else {
                cs0 = append_cos_sin(cache, x.delta, out->cs);
                shift_cs.emplace(x.delta, cs0);
            }
        }
        for (int p = 0; p < n_planes; ++p) {
            KTileItem it;
            std::memset(&it, 0, sizeof(it));
            it.kind = move ? KJOB_TILE : KJOB_STUB;
            it.plane = p;
            it.count = x.count;
            if (move) {
                it.src0 = x.src0;
                it.dst0 = x.src0 + x.delta;
                it.delta = x.delta;
                it.cs = (cs0 >= 0 && planes[p].rot != KROT_NONE) ? cs0 + planes[p].cs_off : -1;
            } else {
                it.dst0 = x.dst0;
                it.stub = static_cast<const char*>(dirs[x.dir].stub[p]);
                it.cs = -1;
            }
            // rotating narrow interleaved bands: tiles of whole packed blocks, units packed
            it.tile_chunks = tile_base;
            const int32_t blk = planes[p].pack_groups * planes[p].tpr;
            if (LEYLINE_TILE_PACK && move && it.cs >= 0 && planes[p].pack_groups && blk <= tile_base) {
                it.tile_chunks = (tile_base / blk) * blk;
                it.pack = 1;
            }
            const int64_t tiles = tile_count(x.count, planes[p].tpr, it.tile_chunks);
            const int64_t tickets = int64_t(cache->n_layers) * tiles;
            it.n_tiles = int32_t(tiles);
            it.ticket0 = int32_t(cur.tickets);
            it.flag0 = -1;
            if (move) {
                it.flag0 = int32_t(n_flags);
                n_flags += tickets;
            }
            for (size_t a = 0; a < cur.items.size(); ++a) {
                const KTileItem& A = cur.items[a];
                if (A.kind == KJOB_TILE && A.plane == p && it.dst0 < A.src0 + A.count && A.src0 < it.dst0 + it.count)
                    it.waits |= 1u << a;
            }
            cur.tickets += tickets;
            if (cur.tickets > INT32_MAX - 1024 || n_flags > INT32_MAX - 1024) return LEYLINE_E_INVAL;
            cur.items.push_back(it);
        }
    }
    if (!cur.items.empty()) out->tile_launches.push_back(std::move(cur));
    out->ws_flags = 256 * int64_t(out->tile_launches.size());
    out->ws_cs = align256(out->ws_flags + 4 * n_flags);
    out->ws_bytes = align256(out->ws_cs + int64_t(sizeof(KCosSin)) * int64_t(out->cs.size()));
    return LEYLINE_OK;
}

}  // namespace

int plan_contig(const leyline_cache* cache, int64_t seq_len, const leyline_directive* dirs,
                int32_t n_dirs, ContigSchedule* out) {
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    int rc = describe_cache(cache, false, planes, &n_planes);
    if (rc) return rc;
    if (seq_len < 0 || seq_len > cache->capacity) return LEYLINE_E_RANGE;
    for (int32_t j = 0; j < n_dirs; ++j)
        if (dirs && dirs[j].seq != 0) return LEYLINE_E_RANGE;
    std::vector<leyline_directive> resolved;
    rc = resolve_forget(dirs, n_dirs, 1, nullptr, seq_len, &resolved, &dirs);
    if (rc) return rc;
    rc = check_sequence(seq_len, dirs, n_dirs, n_planes);
    if (rc) return rc;

    int64_t new_len = seq_len;
    for (int32_t j = 0; j < n_dirs; ++j) {
        if (dirs[j].stub_len > cache->capacity) return LEYLINE_E_CAPACITY;
        new_len += dirs[j].stub_len - (dirs[j].span_end - dirs[j].span_start);
    }
    if (new_len > cache->capacity) return LEYLINE_E_CAPACITY;
    out->new_len = new_len;
    out->launches.clear();
    out->tiles = false;
    out->tile_launches.clear();
    out->cs.clear();
    out->ws_flags = out->ws_cs = out->ws_bytes = 0;

    // Jobs: each downstream segment [e_j, s_{j+1}) moved by its running shift, each stub copied.
    std::vector<ContigJobHost> jobs;
    int64_t shift = 0;
    for (int32_t j = 0; j < n_dirs; ++j) {
        const leyline_directive& d = dirs[j];
        if (d.stub_len > 0)
            jobs.push_back(ContigJobHost{KJOB_STUB, 0, d.span_start + shift, d.stub_len, 0, j});
        shift += d.stub_len - (d.span_end - d.span_start);
        const int64_t seg_end = (j + 1 < n_dirs) ? dirs[j + 1].span_start : seq_len;
        const int64_t count = seg_end - d.span_end;
        if (count > 0 && shift != 0)
            jobs.push_back(ContigJobHost{KJOB_CHAIN, d.span_end, 0, count, shift, j});
    }
    if (jobs.empty()) return LEYLINE_OK;
    // kernels index the chunks of one (job, plane) with 31-bit integers
    for (const ContigJobHost& x : jobs)
        for (int p = 0; p < n_planes; ++p)
            if (x.count * planes[p].row_chunks > INT32_MAX - 2 * int64_t(KTILE_CHUNKS)) return LEYLINE_E_INVAL;

    // Job a must finish before job b when b writes a row that a reads.  The resulting graph is
    // acyclic: a left-moving segment can only wait for segments to its left, a right-moving one
    // only for segments to its right, and a stub only for moves.  The destinations of all jobs
    // are disjoint intervals, and so are the sources of the moves: one sweep over both, sorted by
    // start, meets every overlapping (source, destination) pair, at most one per interval of
    // either list.  A job's level is the length of the longest chain of jobs before it.
    const size_t n = jobs.size();
    auto dst_lo = [&](const ContigJobHost& x) { return x.kind == KJOB_STUB ? x.dst0 : x.src0 + x.delta; };
    std::vector<size_t> by_dst(n), by_src;
    for (size_t k = 0; k < n; ++k) {
        by_dst[k] = k;
        if (jobs[k].kind != KJOB_STUB) by_src.push_back(k);
    }
    std::sort(by_dst.begin(), by_dst.end(), [&](size_t a, size_t b) { return dst_lo(jobs[a]) < dst_lo(jobs[b]); });
    std::sort(by_src.begin(), by_src.end(), [&](size_t a, size_t b) { return jobs[a].src0 < jobs[b].src0; });
    std::vector<std::vector<size_t>> succ(n);
    std::vector<int> indeg(n, 0);
    for (size_t i = 0, j = 0; i < by_dst.size() && j < by_src.size();) {
        const size_t b = by_dst[i], a = by_src[j];
        const int64_t blo = dst_lo(jobs[b]), bhi = blo + jobs[b].count;
        const int64_t alo = jobs[a].src0, ahi = alo + jobs[a].count;
        if (a != b && blo < ahi && alo < bhi) {
            succ[a].push_back(b);
            ++indeg[b];
        }
        if (bhi < ahi) ++i; else ++j;
    }
    std::vector<int> level(n, 0);
    std::vector<size_t> ready;
    for (size_t k = 0; k < n; ++k)
        if (indeg[k] == 0) ready.push_back(k);
    size_t done = 0;
    while (!ready.empty()) {
        const size_t a = ready.back();
        ready.pop_back();
        ++done;
        for (size_t b : succ[a]) {
            level[b] = std::max(level[b], level[a] + 1);
            if (--indeg[b] == 0) ready.push_back(b);
        }
    }
    if (done != n) return LEYLINE_E_INVAL;     // not reached: the graph is acyclic

    const int n_levels = *std::max_element(level.begin(), level.end()) + 1;
    // Ordered tiles need every plane to move single chunks (half-split bands whose partners
    // cannot be exchanged between lanes use ordered chains).
    bool tiles_ok = true;
    int64_t row_bytes_all = 0;
    for (int p = 0; p < n_planes; ++p) {
        if (planes[p].rot == KROT_NEOX && !planes[p].neox_lanes) tiles_ok = false;
        row_bytes_all += planes[p].row_bytes;
    }
    // Within a job, a left shift by m makes row x the destination of row x + m.  Splitting the
    // source range into rounds of at most m rows, taken in ascending order (descending for a
    // right shift), leaves each round with disjoint sources and destinations, and every row a
    // round overwrites was read by an earlier round.  Rounds cost one launch each: they are used
    // for a single round, or when every round moves enough bytes to fill the device.  Once some
    // move would need rounds too small or too many, the whole call runs as ordered tiles.
    bool need_tiles = false;
    for (const ContigJobHost& x : jobs) {
        if (x.kind == KJOB_STUB) continue;
        const int64_t m = x.delta < 0 ? -x.delta : x.delta;
        const int64_t nr = (x.count + m - 1) / m;
        const bool big_rounds = nr == 1 || m * row_bytes_all * cache->n_layers >= ROUND_MIN_BYTES;
        if (nr > MAX_ROUNDS || !big_rounds) need_tiles = true;
    }
    if (tiles_ok && need_tiles) {
        // A call of few full-size tiles cannot fill the device and is bound by each tile's chain
        // of latencies (ticket, loads, flag, stores): it is planned again with quarter-size tiles.
        const size_t cs_before = out->cs.size();
        int rc = plan_tiles(cache, dirs, planes, n_planes, jobs, level, KTILE_CHUNKS, out);
        int64_t tickets = 0;
        for (const TileLaunchHost& tl : out->tile_launches) tickets += tl.tickets;
        if (rc == LEYLINE_OK && tickets < KTILE_SMALL_TICKETS) {
            out->cs.resize(cs_before);
            out->tile_launches.clear();
            rc = plan_tiles(cache, dirs, planes, n_planes, jobs, level, KTILE_SMALL_CHUNKS, out);
        }
        return rc;
    }

    const int32_t cs_need = cos_sin_per_shift(cache);
    for (int lv = 0; lv < n_levels; ++lv) {
        std::vector<std::vector<ContigJobHost>> rounds(1);
        for (size_t a = 0; a < n; ++a) {
            if (level[a] != lv) continue;
            const ContigJobHost& x = jobs[a];
            if (x.kind == KJOB_STUB) {
                rounds[0].push_back(x);
                continue;
            }
            const int64_t m = x.delta < 0 ? -x.delta : x.delta;
            const int64_t nr = (x.count + m - 1) / m;
            if (nr > MAX_ROUNDS) {              // only without tiles: ordered chains
                rounds[0].push_back(x);
                rounds[0].back().kind = KJOB_CHAIN;
                continue;
            }
            if (int64_t(rounds.size()) < nr) rounds.resize(size_t(nr));
            // equal rounds of at most m rows (no small trailing launch)
            const int64_t len = (x.count + nr - 1) / nr;
            for (int64_t r = 0; r < nr; ++r) {
                int64_t lo, hi;
                if (x.delta < 0) {
                    lo = x.src0 + r * len;
                    hi = std::min(x.src0 + x.count, lo + len);
                } else {
                    hi = x.src0 + x.count - r * len;
                    lo = std::max(x.src0, hi - len);
                }
                if (hi <= lo) continue;
                rounds[size_t(r)].push_back(ContigJobHost{KJOB_ROUND, lo, 0, hi - lo, x.delta, x.dir});
            }
        }
        for (const auto& rj : rounds) {
            std::vector<ContigJobHost> cur;
            int32_t cs_used = 0;
            for (const ContigJobHost& x : rj) {
                const int32_t need = x.kind == KJOB_STUB ? 0 : cs_need;
                if (int(cur.size()) == KMAX_JOBS || cs_used + need > KMAX_CS) {
                    out->launches.push_back(cur);
                    cur.clear();
                    cs_used = 0;
                }
                cur.push_back(x);
                cs_used += need;
            }
            if (!cur.empty()) out->launches.push_back(cur);
        }
    }
    return LEYLINE_OK;
}

// ----------------------------------------------------------------------------------- paged --

namespace {

struct Piece {                 // a run of new positions with one source
    int64_t lo, hi;            // new positions [lo, hi)
    bool stub;
    int64_t shift;             // old row = new position - shift
    int32_t dir;               // directive whose segment / stub this is (-1: prefix)
};

}  // namespace

int plan_paged(int32_t page_size, int32_t n_seqs, const int32_t* seq_lens,
               const leyline_directive* dirs, int32_t n_dirs, int32_t n_planes, bool remap,
               PagedPlan* out) {
    if (page_size < 1 || n_seqs < 0 || (n_seqs > 0 && !seq_lens) || n_dirs < 0 ||
        (n_dirs > 0 && !dirs))
        return LEYLINE_E_INVAL;
    for (int32_t b = 0; b < n_seqs; ++b)
        if (seq_lens[b] < 0) return LEYLINE_E_RANGE;
    for (int32_t j = 0; j < n_dirs; ++j) {
        if (dirs[j].seq < 0 || dirs[j].seq >= n_seqs) return LEYLINE_E_RANGE;
        if (j > 0 && dirs[j].seq < dirs[j - 1].seq) return LEYLINE_E_ORDER;
    }
    {
        const int rc = resolve_forget(dirs, n_dirs, n_seqs, seq_lens, 0, &out->resolved, &dirs);
        if (rc) return rc;
    }
    out->dirs = dirs;
    const int64_t P = page_size;
    out->page_size = page_size;
    out->n_seqs = n_seqs;
    out->new_lens.assign(size_t(n_seqs), 0);
    out->run_begin.assign(size_t(n_seqs) + 1, 0);
    out->runs.clear();
    out->freed.clear();
    int64_t n_fresh = 0, n_remap = 0, n_freed = 0;

    int32_t j0 = 0;
    std::vector<Piece> pieces;
    std::vector<std::pair<int64_t, int64_t>> kept;   // re-used old pages [lo, hi), ascending
    for (int32_t b = 0; b < n_seqs; ++b) {
        int32_t j1 = j0;
        while (j1 < n_dirs && dirs[j1].seq == b) ++j1;
        const int64_t n = seq_lens[b];
        int rc = check_sequence(n, dirs + j0, j1 - j0, n_planes);
        if (rc) return rc;
        // Pieces in new-position order.  Adjacent old-row pieces with the same shift (around a
        // directive that deletes and inserts nothing) are one piece: the page rule looks at rows.
        pieces.clear();
        auto add = [&](const Piece& p) {
            if (!p.stub && !pieces.empty()) {
                Piece& q = pieces.back();
                if (!q.stub && q.hi == p.lo && q.shift == p.shift) {
                    q.hi = p.hi;
                    q.dir = p.dir;
                    return;
                }
            }
            pieces.push_back(p);
        };
        int64_t shift = 0, cursor = 0, pos = 0;
        for (int32_t j = j0; j < j1; ++j) {
            const leyline_directive& d = dirs[j];
            if (d.span_start > cursor) {
                add(Piece{pos, pos + d.span_start - cursor, false, shift, j > j0 ? j - 1 : -1});
                pos += d.span_start - cursor;
            }
            if (d.stub_len > 0) {
                add(Piece{pos, pos + d.stub_len, true, 0, j});
                pos += d.stub_len;
            }
            shift += d.stub_len - (d.span_end - d.span_start);
            cursor = d.span_end;
            if (pos > INT32_MAX) return LEYLINE_E_CAPACITY;
        }
        if (n > cursor) {
            add(Piece{pos, pos + n - cursor, false, shift, j1 > j0 ? j1 - 1 : -1});
            pos += n - cursor;
        }
        if (pos > INT32_MAX) return LEYLINE_E_CAPACITY;
        const int64_t n_new = pos;
        out->new_lens[size_t(b)] = int32_t(n_new);
        const int64_t old_pages = (n + P - 1) / P;
        const int64_t new_pages = (n_new + P - 1) / P;
        out->run_begin[size_t(b)] = int32_t(out->runs.size());
        // A new page is re-used (IDENTITY for shift 0, REMAP for another multiple of the page
        // size) when all its valid rows lie in one old-row piece whose shift keeps in-page
        // offsets; every other page is ASSEMBLE.
        auto assemble = [&](int64_t k0, int64_t k1) {
            if (k1 <= k0) return;
            out->runs.push_back(KPageRun{b, int32_t(k0), int32_t(k1 - k0), LEYLINE_PAGE_ASSEMBLE,
                                         int32_t(n_fresh), int32_t(n_fresh), -1, 0});
            n_fresh += k1 - k0;
        };
        kept.clear();
        int64_t kcur = 0;
        for (const Piece& p : pieces) {
            if (p.stub || p.shift % P != 0 || (p.shift != 0 && !remap)) continue;
            const int64_t first = (p.lo + P - 1) / P;
            const int64_t last = p.hi == n_new ? (p.hi + P - 1) / P : p.hi / P;
            if (first >= last) continue;
            assemble(kcur, first);
            const int64_t src0 = first - p.shift / P;
            if (p.shift == 0) {
                out->runs.push_back(KPageRun{b, int32_t(first), int32_t(last - first), LEYLINE_PAGE_IDENTITY,
                                             int32_t(src0), 0, -1, 0});
            } else {
                out->runs.push_back(KPageRun{b, int32_t(first), int32_t(last - first), LEYLINE_PAGE_REMAP,
                                             int32_t(src0), int32_t(n_remap), p.dir, 0});
                n_remap += last - first;
            }
            kept.emplace_back(src0, src0 + (last - first));
            kcur = last;
        }
        assemble(kcur, new_pages);
        int64_t c = 0;
        for (const auto& r : kept) {
            if (r.first > c) {
                out->freed.push_back(KFreedRun{b, int32_t(c), int32_t(r.first - c), int32_t(n_freed)});
                n_freed += r.first - c;
            }
            c = r.second;
        }
        if (old_pages > c) {
            out->freed.push_back(KFreedRun{b, int32_t(c), int32_t(old_pages - c), int32_t(n_freed)});
            n_freed += old_pages - c;
        }
        if (n_fresh > INT32_MAX || n_remap > INT32_MAX || n_freed > INT32_MAX) return LEYLINE_E_CAPACITY;
        j0 = j1;
    }
    out->run_begin[size_t(n_seqs)] = int32_t(out->runs.size());
    out->n_fresh = int32_t(n_fresh);
    out->n_remap = int32_t(n_remap);
    out->n_freed = int32_t(n_freed);
    return LEYLINE_OK;
}

int build_paged_image(const leyline_cache* cache, const PagedPlan& plan, int32_t n_seqs,
                      const leyline_directive* dirs, int32_t n_dirs, int32_t bt_stride,
                      PagedImage* img) {
    std::vector<KSeqEntry> seqs(static_cast<size_t>(n_seqs));
    std::vector<KDirEntry> dtab(static_cast<size_t>(n_dirs));
    std::vector<KCosSin> cs;
    const bool any_rot = cos_sin_per_shift(cache) > 0;
    int32_t j0 = 0;
    for (int32_t b = 0; b < n_seqs; ++b) {
        int32_t j1 = j0;
        while (j1 < n_dirs && dirs[j1].seq == b) ++j1;
        KSeqEntry& e = seqs[size_t(b)];
        std::memset(&e, 0, sizeof(e));
        e.dir_begin = j0;
        e.dir_count = j1 - j0;
        e.new_len = plan.new_lens[size_t(b)];
        e.run_begin = plan.run_begin[size_t(b)];
        e.run_count = plan.run_begin[size_t(b) + 1] - plan.run_begin[size_t(b)];
        int64_t shift = 0;
        for (int32_t j = j0; j < j1; ++j) {
            const leyline_directive& d = dirs[j];
            KDirEntry& de = dtab[size_t(j)];
            std::memset(&de, 0, sizeof(de));
            de.stub_start = d.span_start + shift;
            de.stub_len = d.stub_len;
            shift += d.stub_len - (d.span_end - d.span_start);
            de.delta = shift;
            de.cs = (shift != 0 && any_rot) ? append_cos_sin(cache, shift, cs) : -1;
            for (int p = 0; p < cache->n_planes; ++p)
                de.stub[p] = static_cast<const char*>(d.stub[p]);
        }
        j0 = j1;
    }
    std::vector<KPageRun> asm_runs, remap_runs;
    for (const KPageRun& r : plan.runs) {
        if (r.k0 + r.count > bt_stride) return LEYLINE_E_CAPACITY;
        if (r.kind == LEYLINE_PAGE_ASSEMBLE) asm_runs.push_back(r);
        else if (r.kind == LEYLINE_PAGE_REMAP) remap_runs.push_back(r);
    }

    KPagedTables& t = img->tables;
    std::memset(&t, 0, sizeof(t));
    int64_t off = 0;
    auto place = [&](size_t bytes, int64_t align) {
        off = (off + align - 1) / align * align;
        const int64_t at = off;
        off += int64_t(bytes);
        return at;
    };
    // the plan tables, packed (16-byte aligned) so that small plans fit in kernel arguments
    t.off_seq = place(seqs.size() * sizeof(KSeqEntry), 16);
    t.off_dir = place(dtab.size() * sizeof(KDirEntry), 16);
    t.off_cs = place(cs.size() * sizeof(KCosSin), 16);
    t.off_runs = place(plan.runs.size() * sizeof(KPageRun), 16);
    t.off_asm_runs = place(asm_runs.size() * sizeof(KPageRun), 16);
    t.off_remap_runs = place(remap_runs.size() * sizeof(KPageRun), 16);
    t.off_freed_runs = place(plan.freed.size() * sizeof(KFreedRun), 16);
    t.upload = (off + 15) / 16 * 16;
    const int64_t n_rows = int64_t(plan.n_fresh) * plan.page_size;
    if (n_rows > INT32_MAX) return LEYLINE_E_CAPACITY;
    // the tables the kernels write: the row table (and its destination order) of a large gather
    const bool row_table = n_rows > KINLINE_ROWS;
    t.off_rows = place(row_table ? size_t(n_rows) * sizeof(KRowMove) : 0, 256);
    t.off_order = place(row_table && plan.n_fresh >= KORDER_MIN ? size_t(plan.n_fresh) * sizeof(int32_t) : 0, 256);
    // the REMAP pages in physical order, when some plane rotates wide bands
    int64_t rot_row_bytes = 0;
    for (int p = 0; p < cache->n_planes; ++p)
        rot_row_bytes = std::max<int64_t>(rot_row_bytes, int64_t(cache->planes[p].n_heads) *
                                                             cache->planes[p].rot_dim * elem_size(cache->dtype));
    const bool remap_sorted = plan.n_remap >= KORDER_MIN && rot_row_bytes >= KREMAP_SORT_BYTES;
    t.off_remap_sorted = place(remap_sorted ? size_t(plan.n_remap) * sizeof(KRemapPage) : 0, 256);
    t.total = (off + 255) / 256 * 256;
    t.n_seqs = n_seqs; t.n_dirs = n_dirs; t.n_cs = int32_t(cs.size());
    t.n_runs = int32_t(plan.runs.size());
    t.n_asm_runs = int32_t(asm_runs.size());
    t.n_remap_runs = int32_t(remap_runs.size());
    t.n_freed_runs = int32_t(plan.freed.size());
    t.n_asm = plan.n_fresh; t.n_remap = plan.n_remap; t.n_freed = plan.n_freed;
    t.bt_stride = bt_stride;
    t.n_rows = int32_t(n_rows);
    t.remap_sorted = remap_sorted ? 1 : 0;
    img->bytes.assign(size_t(t.upload), 0);
    auto put = [&](int64_t at, const void* src, size_t bytes) {
        if (bytes) std::memcpy(img->bytes.data() + at, src, bytes);
    };
    put(t.off_seq, seqs.data(), seqs.size() * sizeof(KSeqEntry));
    put(t.off_dir, dtab.data(), dtab.size() * sizeof(KDirEntry));
    put(t.off_cs, cs.data(), cs.size() * sizeof(KCosSin));
    put(t.off_runs, plan.runs.data(), plan.runs.size() * sizeof(KPageRun));
    put(t.off_asm_runs, asm_runs.data(), asm_runs.size() * sizeof(KPageRun));
    put(t.off_remap_runs, remap_runs.data(), remap_runs.size() * sizeof(KPageRun));
    put(t.off_freed_runs, plan.freed.data(), plan.freed.size() * sizeof(KFreedRun));
    return LEYLINE_OK;
}

int check_table_width(const PagedPlan& plan, const int32_t* seq_lens, int32_t bt_stride) {
    for (int32_t b = 0; b < plan.n_seqs; ++b) {
        const int64_t old_pages = (int64_t(seq_lens[b]) + plan.page_size - 1) / plan.page_size;
        const int64_t new_pages = (int64_t(plan.new_lens[size_t(b)]) + plan.page_size - 1) / plan.page_size;
        if (old_pages > bt_stride || new_pages > bt_stride) return LEYLINE_E_CAPACITY;
    }
    return LEYLINE_OK;
}

}  // namespace leyline

// ------------------------------------------------------------------------ host-only C ABI ---

extern "C" const char* leyline_strerror(int code) {
    switch (code) {
        case LEYLINE_OK: return "ok";
        case LEYLINE_E_INVAL: return "invalid argument or cache layout";
        case LEYLINE_E_RANGE: return "span or sequence index out of range";
        case LEYLINE_E_ORDER: return "directives not sorted by (seq, span_start)";
        case LEYLINE_E_OVERLAP: return "directive spans overlap";
        case LEYLINE_E_CAPACITY: return "capacity exceeded (rows, pages, block table or freed list)";
        case LEYLINE_E_MODE: return "a FORGET directive must be the last of its sequence and carry no replacement";
        case LEYLINE_E_WORKSPACE: return "workspace missing or too small";
        case LEYLINE_E_HIP: return "HIP runtime error";
        default: return "unknown leyline status";
    }
}

extern "C" int leyline_abi_version(void) { return LEYLINE_ABI_VERSION; }

extern "C" int leyline_paged_query(const leyline_cache* cache, int32_t n_seqs,
                                   const int32_t* seq_lens, int32_t bt_stride,
                                   const leyline_directive* dirs, int32_t n_dirs, uint32_t flags,
                                   int32_t* new_seq_lens, int32_t* n_fresh_needed, int32_t* n_freed,
                                   int64_t* workspace_bytes) {
    using namespace leyline;
    KPlane planes[LEYLINE_MAX_PLANES];
    int n_planes = 0;
    int rc = describe_cache(cache, true, planes, &n_planes);
    if (rc) return rc;
    if (bt_stride < 0) return LEYLINE_E_INVAL;
    if (flags & ~uint32_t(LEYLINE_PAGED_COPY_ON_WRITE)) return LEYLINE_E_INVAL;
    PagedPlan plan;
    rc = plan_paged(cache->page_size, n_seqs, seq_lens, dirs, n_dirs, n_planes,
                    !(flags & LEYLINE_PAGED_COPY_ON_WRITE), &plan);
    if (rc) return rc;
    rc = check_table_width(plan, seq_lens, bt_stride);
    if (rc) return rc;
    PagedImage img;
    rc = build_paged_image(cache, plan, n_seqs, plan.dirs, n_dirs, bt_stride, &img);
    if (rc) return rc;
    if (new_seq_lens)
        for (int32_t b = 0; b < n_seqs; ++b) new_seq_lens[b] = plan.new_lens[size_t(b)];
    if (n_fresh_needed) *n_fresh_needed = plan.n_fresh;
    if (n_freed) *n_freed = plan.n_freed;
    if (workspace_bytes) *workspace_bytes = img.tables.total;
    return LEYLINE_OK;
}

extern "C" int leyline_paged_plan(int32_t page_size, int32_t n_seqs, const int32_t* seq_lens,
                                  const leyline_directive* dirs, int32_t n_dirs, uint32_t flags,
                                  int32_t bt_stride,
                                  int32_t* kind_out, int32_t* src_out,
                                  int32_t* freed_seq_out, int32_t* freed_page_out, int32_t freed_cap) {
    using namespace leyline;
    if (bt_stride < 0 || (n_seqs > 0 && (!kind_out || !src_out))) return LEYLINE_E_INVAL;
    if (flags & ~uint32_t(LEYLINE_PAGED_COPY_ON_WRITE)) return LEYLINE_E_INVAL;
    PagedPlan plan;
    // stub pointers are not needed for a symbolic plan: validate them against zero planes
    int rc = plan_paged(page_size, n_seqs, seq_lens, dirs, n_dirs, 0,
                        !(flags & LEYLINE_PAGED_COPY_ON_WRITE), &plan);
    if (rc) return rc;
    rc = check_table_width(plan, seq_lens, bt_stride);
    if (rc) return rc;
    if (plan.n_freed > freed_cap) return LEYLINE_E_CAPACITY;
    if (plan.n_freed > 0 && (!freed_seq_out || !freed_page_out)) return LEYLINE_E_INVAL;
    for (int64_t i = 0; i < int64_t(n_seqs) * bt_stride; ++i) {
        kind_out[i] = LEYLINE_PAGE_NONE;
        src_out[i] = -1;
    }
    for (const KPageRun& r : plan.runs)
        for (int32_t c = 0; c < r.count; ++c) {
            const int64_t at = int64_t(r.seq) * bt_stride + r.k0 + c;
            kind_out[at] = r.kind;
            src_out[at] = r.src0 + c;
        }
    for (const KFreedRun& r : plan.freed)
        for (int32_t c = 0; c < r.count; ++c) {
            freed_seq_out[r.out0 + c] = r.seq;
            freed_page_out[r.out0 + c] = r.page0 + c;
        }
    return LEYLINE_OK;
}
