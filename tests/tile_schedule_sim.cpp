// Host-side check of the ordered-tile schedules of contiguous splices.
//
// Random multi-directive splices are planned with the library's planner; every tile launch of a
// plan is then executed on the CPU the way the tile kernel runs it: workgroups take tickets in
// order (at most W in flight), each loads its source chunks, publishes "source read" (moves),
// waits for the flags that tile_wait_flags lists and stores.  The order in which in-flight
// workgroups load and store is drawn at random.  The check fails if a load sees a row that was
// already overwritten, if a wait names a flag outside the launch or of a later ticket, if a
// schedule stalls, or if the rows [0, new_len) differ from the splice's definition (prefix
// unchanged, replacements at s_j + delta_{j-1}, segment j shifted by delta_j).  Values are row
// identities, not data: rotation is not simulated.
//
// The kernel's wait is bounded (tile_wait_bounded, KTILE_SPIN_LIMIT polls): when every in-flight
// tile is blocked, each waiting tile polls until the bound, gives up, flags the timeout status
// and exits without storing.  A correct schedule never gets there.  With PLANT = 1 the first
// move tile of every launch also waits for the flag of the launch's last move tile (a later
// ticket: a planted schedule fault); then the give-up path must let every workgroup exit and
// raise the status bit whenever the fault blocked the launch.
//
// Usage: tile_schedule_sim SEED CASES [PLANT [PERSIST]]
//        (prints "ok <tile cases> <tiles stored> <waits given up>" on success)
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "plan.hpp"

using namespace leyline;

namespace {

struct Shape {
    const char* name;
    int32_t dtype;
    int n_planes;
    int32_t row_elems[2];
    int32_t n_heads[2], head_stride[2], rot_offset[2], rot_dim[2], style[2];
    int64_t max_len;
};

const Shape kShapes[] = {
    // 32-byte rows (2 chunks), an interleaved 8-element band
    {"tiny_interleaved", LEYLINE_BF16, 1, {16, 0}, {1, 0}, {16, 0}, {8, 0}, {8, 0}, {LEYLINE_ROPE_INTERLEAVED, 0}, 30000},
    // K (two heads, half-split bands exchanged between lanes) and V planes, 8 chunks per row
    {"small_kv", LEYLINE_BF16, 2, {64, 64}, {2, 1}, {32, 64}, {0, 0}, {32, 0}, {LEYLINE_ROPE_NEOX, 0}, 8000},
    // MLA rows: c_kv 512 + k_pe 64 bf16 (72 chunks)
    {"mla", LEYLINE_BF16, 1, {576, 0}, {1, 0}, {576, 0}, {512, 0}, {64, 0}, {LEYLINE_ROPE_INTERLEAVED, 0}, 2500},
    // fp32 rows of 4 chunks, no rotary band
    {"f32_plain", LEYLINE_F32, 1, {16, 0}, {1, 0}, {16, 0}, {0, 0}, {0, 0}, {0, 0}, 15000},
};

int64_t orig_val(int p, int l, int64_t row, int64_t c) { return ((((int64_t(p) * 4 + l) << 24) | row) << 10 | c) + 1; }
int64_t stub_val(int j, int p, int l, int64_t t, int64_t c) {
    return -(((((int64_t(j) * 4 + p) * 4 + l) << 24 | t) << 10 | c) + 1);
}

int fail(const char* what, int case_id) {
    std::printf("FAIL case %d: %s\n", case_id, what);
    return 1;
}

}  // namespace

int main(int argc, char** argv) {
    const unsigned seed = argc > 1 ? unsigned(std::atoi(argv[1])) : 1u;
    const int cases = argc > 2 ? std::atoi(argv[2]) : 100;
    const bool plant = argc > 3 && std::atoi(argv[3]) != 0;
    // PERSIST: 0 one tile per workgroup, 1 persistent workgroups, 2 either, drawn per launch
    const int persist_mode = argc > 4 ? std::atoi(argv[4]) : 2;
    int64_t gave_up = 0;
    std::mt19937_64 rng(seed);
    auto uni = [&](int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); };
    int tile_cases = 0;
    int64_t tiles_run = 0;
    for (int ci = 0; ci < cases; ++ci) {
        const Shape& sh = kShapes[uni(0, 3)];
        const int L = int(uni(1, 3));
        const int64_t n = uni(1, sh.max_len);
        // directives: sorted, non-overlapping (adjacent allowed) spans; short shifts are common
        const int k = int(uni(0, 3) == 0 ? uni(9, 48) : uni(1, 8));   // some calls with many directives
        std::vector<int64_t> cuts;
        for (int i = 0; i < 2 * k; ++i) cuts.push_back(uni(0, n));
        std::sort(cuts.begin(), cuts.end());
        std::vector<leyline_directive> dirs(static_cast<size_t>(k));
        int64_t shift = 0, grow = 0;
        for (int j = 0; j < k; ++j) {
            leyline_directive& d = dirs[size_t(j)];
            std::memset(&d, 0, sizeof(d));
            d.span_start = cuts[size_t(2 * j)];
            d.span_end = std::min(cuts[size_t(2 * j + 1)], d.span_start + (uni(0, 3) == 0 ? n : uni(0, 64)));
            if (d.span_end < d.span_start) d.span_end = d.span_start;
            const int64_t span = d.span_end - d.span_start;
            const int pick = int(uni(0, 4));
            d.stub_len = pick == 0 ? 0 : pick == 1 ? span + uni(-3, 3) : pick == 2 ? span : uni(0, 2 * span + 3);
            if (d.stub_len < 0) d.stub_len = 0;
            for (int p = 0; p < sh.n_planes; ++p)
                d.stub[p] = d.stub_len ? reinterpret_cast<const void*>(uintptr_t(0x1000000) * (j + 1) + 0x10000 * p) : nullptr;
            shift += d.stub_len - span;
            grow = std::max(grow, shift);
        }
        const int64_t new_len = n + shift, cap = n + grow + uni(0, 3);
        leyline_cache cache;
        std::memset(&cache, 0, sizeof(cache));
        cache.dtype = sh.dtype;
        cache.n_layers = L;
        cache.n_planes = sh.n_planes;
        cache.capacity = cap;
        for (int p = 0; p < sh.n_planes; ++p) {
            leyline_plane& pl = cache.planes[p];
            pl.base = reinterpret_cast<void*>(uintptr_t(0x100000000ull) * (p + 1));
            pl.row_elems = sh.row_elems[p];
            pl.token_stride = sh.row_elems[p];
            pl.layer_stride = cap * sh.row_elems[p];
            pl.n_heads = sh.n_heads[p];
            pl.head_stride = sh.head_stride[p];
            pl.rot_offset = sh.rot_offset[p];
            pl.rot_dim = sh.rot_dim[p];
            pl.rope_style = sh.style[p];
            pl.rope_base = 10000.0;
        }
        ContigSchedule sched;
        const int rc = plan_contig(&cache, n, dirs.data(), k, &sched);
        if (rc) {
            std::printf("FAIL case %d: plan_contig returned %d\n", ci, rc);
            return 1;
        }
        if (sched.new_len != new_len) return fail("new length", ci);
        if (!sched.tiles) continue;
        ++tile_cases;
        KPlane planes[LEYLINE_MAX_PLANES];
        int n_planes = 0;
        if (describe_cache(&cache, false, planes, &n_planes)) return fail("describe_cache", ci);
        // memory: per plane and layer, cap rows of tpr chunks holding row identities
        std::vector<std::vector<int64_t>> mem(static_cast<size_t>(n_planes * L));
        for (int p = 0; p < n_planes; ++p)
            for (int l = 0; l < L; ++l) {
                auto& m = mem[size_t(p * L + l)];
                const int64_t tpr = planes[p].tpr;
                m.assign(size_t(cap * tpr), 0);
                for (int64_t r = 0; r < cap; ++r)
                    for (int64_t c = 0; c < tpr; ++c) m[size_t(r * tpr + c)] = orig_val(p, l, r, c);
            }
        int64_t n_flags = 0;
        for (const auto& tl : sched.tile_launches)
            for (const auto& it : tl.items)
                if (it.kind == KJOB_TILE) n_flags = std::max<int64_t>(n_flags, it.flag0 + int64_t(L) * it.n_tiles);
        std::vector<int> flags(static_cast<size_t>(n_flags), 0);
        int32_t status = 0;
        for (const auto& tl : sched.tile_launches) {
            if (tl.items.empty() || tl.items.size() > size_t(KTILE_MAX_ITEMS)) return fail("item count", ci);
            KTileParams P;
            std::memset(&P, 0, sizeof(P));
            std::memcpy(P.planes, planes, sizeof(KPlane) * size_t(n_planes));
            std::copy(tl.items.begin(), tl.items.end(), P.items);
            P.n_items = int32_t(tl.items.size());
            P.n_tickets = int32_t(tl.tickets);
            tile_fill_ticket_table(P);
            // ticket -> (item, layer, order); flag -> ticket, for flags of this launch
            struct Tile { int item, layer, order; };
            std::vector<Tile> tiles(static_cast<size_t>(tl.tickets));
            std::vector<int64_t> flag_ticket(size_t(n_flags), -1);
            for (int i = 0; i < P.n_items; ++i) {
                const KTileItem& I = P.items[i];
                if (i + 1 < P.n_items && P.items[i + 1].ticket0 != I.ticket0 + int64_t(L) * I.n_tiles)
                    return fail("ticket ranges", ci);
                if (I.waits >> i) return fail("an item waits for itself or a later item", ci);
                for (int l = 0; l < L; ++l)
                    for (int o = 0; o < I.n_tiles; ++o) {
                        const int64_t t = I.ticket0 + int64_t(l) * I.n_tiles + o;
                        if (tile_item_of(P, int32_t(t)) != i) return fail("ticket to item lookup", ci);
                        tiles[size_t(t)] = Tile{i, l, o};
                        if (I.kind == KJOB_TILE) flag_ticket[size_t(I.flag0 + int64_t(l) * I.n_tiles + o)] = t;
                    }
            }
            // loads and stores of one tile
            auto chunks = [&](const Tile& T, int64_t* g0, int64_t* g1) {
                const KTileItem& I = P.items[T.item];
                const int64_t tpr = planes[I.plane].tpr, total = I.count * tpr;
                const int64_t q = I.delta <= 0 ? T.order : I.n_tiles - 1 - T.order;
                *g0 = q * I.tile_chunks;
                *g1 = std::min(total, *g0 + I.tile_chunks);
            };
            const bool persist = persist_mode == 1 || (persist_mode == 2 && uni(0, 1) == 1);
            std::vector<std::vector<int64_t>> buf(size_t(tl.tickets));
            std::vector<int> state(size_t(tl.tickets), 0);        // 0 taken, 1 loaded, 2 stored
            const int64_t W = std::vector<int64_t>{1, 2, 3, 8, 64, int64_t(1) << 40}[size_t(uni(0, 5))];
            int64_t next = 0;
            std::vector<int64_t> live;
            std::vector<int64_t> waits;
            // planted fault: the first move tile also waits for the last move tile's flag
            int64_t victim = -1, planted = -1;
            if (plant) {
                for (int64_t t = 0; t < tl.tickets; ++t)
                    if (P.items[tiles[size_t(t)].item].kind == KJOB_TILE) {
                        const Tile& T = tiles[size_t(t)];
                        const KTileItem& I = P.items[T.item];
                        const int64_t f = I.flag0 + int64_t(T.layer) * I.n_tiles + T.order;
                        if (victim < 0) victim = t;
                        else planted = f;
                    }
                if (planted < 0) victim = -1;
            }
            // whether loaded tile t may store (every flag it waits for set); bad: a wait names a
            // flag outside the launch or of a later ticket
            auto ready_to_store = [&](int64_t t, bool* bad) {
                const Tile& T = tiles[size_t(t)];
                bool ready = true;
                tile_wait_flags(P, T.item, T.layer, T.order, [&](int64_t f) {
                    if (f < 0 || f >= n_flags || flag_ticket[size_t(f)] < 0 || flag_ticket[size_t(f)] >= t) *bad = true;
                    else if (!flags[size_t(f)]) ready = false;
                });
                if (t == victim && !flags[size_t(planted)]) ready = false;
                return ready;
            };
            // reads tile t's chunks into buf[t] (0, or 1: a load saw an overwritten row, 2: unknown
            // replacement); publish(t) sets a move tile's "source read" flag; store_tile writes
            auto load_tile = [&](int64_t t) -> int {
                const Tile& T = tiles[size_t(t)];
                const KTileItem& I = P.items[T.item];
                const int p = I.plane;
                const int64_t tpr = planes[p].tpr;
                auto& m = mem[size_t(p * L + T.layer)];
                int64_t g0, g1;
                chunks(T, &g0, &g1);
                auto& b = buf[size_t(t)];
                b.resize(size_t(g1 - g0));
                for (int64_t g = g0; g < g1; ++g) {
                    int32_t r32, c32;             // the kernel's unit layout (packed or not)
                    row_unit(planes[p], LEYLINE_TILE_PACK && I.pack, int32_t(g), I.count, r32, c32);
                    const int64_t r = r32, c = c32;
                    if (I.kind == KJOB_TILE) {
                        const int64_t v = m[size_t((I.src0 + r) * tpr + c)];
                        if (v != orig_val(p, T.layer, I.src0 + r, c)) return 1;
                        b[size_t(g - g0)] = v;
                    } else {
                        int j = -1;
                        for (int jj = 0; jj < k; ++jj)
                            if (dirs[size_t(jj)].stub[p] == I.stub) j = jj;
                        if (j < 0) return 2;
                        b[size_t(g - g0)] = stub_val(j, p, T.layer, r, c);
                    }
                }
                return 0;
            };
            auto publish = [&](int64_t t) {
                const Tile& T = tiles[size_t(t)];
                const KTileItem& I = P.items[T.item];
                if (I.kind == KJOB_TILE) flags[size_t(I.flag0 + int64_t(T.layer) * I.n_tiles + T.order)] = 1;
            };
            auto store_tile = [&](int64_t t) {
                const Tile& T = tiles[size_t(t)];
                const KTileItem& I = P.items[T.item];
                const int p = I.plane;
                const int64_t tpr = planes[p].tpr;
                auto& m = mem[size_t(p * L + T.layer)];
                int64_t g0, g1;
                chunks(T, &g0, &g1);
                const auto& b = buf[size_t(t)];
                for (int64_t g = g0; g < g1; ++g) {
                    int32_t r32, c32;             // the kernel's unit layout (packed or not)
                    row_unit(planes[p], LEYLINE_TILE_PACK && I.pack, int32_t(g), I.count, r32, c32);
                    const int64_t r = r32, c = c32;
                    m[size_t((I.dst0 + r) * tpr + c)] = b[size_t(g - g0)];
                }
                ++tiles_run;
            };
            auto load_fail = [&](int rc) {
                return fail(rc == 1 ? "a load saw an overwritten row" : "unknown replacement", ci);
            };
            if (persist) {
                // G persistent workgroups (the kernel's LEYLINE_TILE_PERSIST design): each takes a
                // ticket, loads it, then repeatedly publishes its current tile and takes the next
                // ticket, loads the next tile (the load may complete before or after the store
                // below), waits for the current tile's flags and stores it
                struct Wg { int phase; int64_t cur, nxt; bool nxt_loaded; };
                const int64_t G = std::vector<int64_t>{1, 2, 3, 8, 64}[size_t(uni(0, 4))];
                std::vector<Wg> wgs(size_t(G), Wg{0, -1, -1, false});
                size_t done = 0;
                while (done < wgs.size()) {
                    // enabled actions: (workgroup, kind) with kind 0 take first ticket, 1 load the
                    // current tile, 2 publish + take next, 3 load the next tile, 4 store current
                    std::vector<std::pair<size_t, int>> acts;
                    for (size_t w = 0; w < wgs.size(); ++w) {
                        const Wg& g = wgs[w];
                        if (g.phase == 0) acts.emplace_back(w, 0);
                        else if (g.phase == 1) acts.emplace_back(w, 1);
                        else if (g.phase == 2) acts.emplace_back(w, 2);
                        else if (g.phase == 3 || g.phase == 4) {
                            if (g.nxt >= 0 && !g.nxt_loaded) acts.emplace_back(w, 3);
                            if (g.phase == 3) {
                                bool bad = false;
                                const bool ready = ready_to_store(g.cur, &bad);
                                if (bad) return fail("a wait names a flag outside the launch or of a later ticket", ci);
                                if (ready) acts.emplace_back(w, 4);
                            }
                        }
                    }
                    // a workgroup whose current tile is stored (or given up) moves on once its next
                    // tile is loaded, or exits when there is none
                    auto move_on = [&](Wg& g) {
                        if (g.phase == 4 && (g.nxt < 0 || g.nxt_loaded)) {
                            if (g.nxt < 0) { g.phase = 5; ++done; }
                            else { g.cur = g.nxt; g.nxt = -1; g.phase = 2; }
                        }
                    };
                    if (acts.empty()) {
                        if (!plant) return fail("persistent schedule stalled", ci);
                        // every workgroup is blocked in its wait: each gives up (bounded wait),
                        // stores nothing and goes on
                        int blocked = 0;
                        for (Wg& g : wgs) {
                            if (g.phase != 3) continue;
                            ++blocked;
                            bool bad = false;
                            int64_t polls = 0;
                            const bool ok = tile_wait_bounded([&] { return ready_to_store(g.cur, &bad); },
                                                              [&] { ++polls; }, KTILE_SPIN_LIMIT);
                            if (ok || polls != KTILE_SPIN_LIMIT) return fail("bounded wait", ci);
                            status |= LEYLINE_STATUS_TILE_TIMEOUT;
                            ++gave_up;
                            g.phase = 4;
                            move_on(g);
                        }
                        if (!blocked) return fail("persistent workgroups blocked outside their wait", ci);
                        continue;
                    }
                    const auto a = acts[size_t(uni(0, int64_t(acts.size()) - 1))];
                    Wg& g = wgs[a.first];
                    switch (a.second) {
                    case 0:
                        if (next >= tl.tickets) { g.phase = 5; ++done; break; }
                        g.cur = next++;
                        g.phase = 1;
                        break;
                    case 1:
                        if (int rc = load_tile(g.cur)) return load_fail(rc);
                        g.phase = 2;
                        break;
                    case 2:
                        publish(g.cur);
                        g.nxt = next < tl.tickets ? next++ : -1;
                        g.nxt_loaded = false;
                        g.phase = 3;
                        break;
                    case 3:
                        if (int rc = load_tile(g.nxt)) return load_fail(rc);
                        g.nxt_loaded = true;
                        break;
                    case 4:
                        store_tile(g.cur);
                        g.phase = 4;
                        break;
                    }
                    move_on(g);
                }
                continue;
            }
            while (next < tl.tickets || !live.empty()) {
                // possible actions: take the next ticket, load a taken tile, store a loaded one
                std::vector<std::pair<int, int64_t>> acts;
                if (next < tl.tickets && int64_t(live.size()) < W) acts.emplace_back(0, next);
                for (int64_t t : live) {
                    if (state[size_t(t)] == 0) {
                        acts.emplace_back(1, t);
                        continue;
                    }
                    bool bad = false;
                    const bool ready = ready_to_store(t, &bad);
                    if (bad) return fail("a wait names a flag outside the launch or of a later ticket", ci);
                    if (ready) acts.emplace_back(2, t);
                }
                if (acts.empty()) {
                    // every in-flight tile is blocked: nothing changes while they poll, so each
                    // waits out its bound, flags the timeout and exits without storing
                    if (!plant) return fail("schedule stalled", ci);
                    std::vector<int64_t> blocked = live;
                    for (int64_t t : blocked) {
                        bool bad = false;
                        int64_t polls = 0;
                        const bool ok = tile_wait_bounded([&] { return ready_to_store(t, &bad); },
                                                          [&] { ++polls; }, KTILE_SPIN_LIMIT);
                        if (ok || polls != KTILE_SPIN_LIMIT) return fail("bounded wait", ci);
                        status |= LEYLINE_STATUS_TILE_TIMEOUT;
                        state[size_t(t)] = 2;
                        live.erase(std::find(live.begin(), live.end(), t));
                        ++gave_up;
                    }
                    continue;
                }
                const auto a = acts[size_t(uni(0, int64_t(acts.size()) - 1))];
                const int64_t t = a.second;
                if (a.first == 0) {
                    live.push_back(t);
                    ++next;
                    continue;
                }
                if (a.first == 1) {
                    if (int rc = load_tile(t)) return load_fail(rc);
                    publish(t);
                    state[size_t(t)] = 1;
                } else {
                    store_tile(t);
                    state[size_t(t)] = 2;
                    live.erase(std::find(live.begin(), live.end(), t));
                }
            }
        }
        // every workgroup has exited; a launch that gave up leaves its rows unspecified
        if (status) continue;
        // rows [0, new_len) against the definition
        for (int p = 0; p < n_planes; ++p)
            for (int l = 0; l < L; ++l) {
                const auto& m = mem[size_t(p * L + l)];
                const int64_t tpr = planes[p].tpr;
                auto check_row = [&](int64_t pos, int j, int64_t src) -> bool {   // j >= 0: stub j row src
                    for (int64_t c = 0; c < tpr; ++c) {
                        const int64_t want = j >= 0 ? stub_val(j, p, l, src, c) : orig_val(p, l, src, c);
                        if (m[size_t(pos * tpr + c)] != want) return false;
                    }
                    return true;
                };
                int64_t pos = 0, delta = 0;
                for (int64_t r = 0; r < dirs[0].span_start; ++r, ++pos)
                    if (!check_row(pos, -1, r)) return fail("prefix row", ci);
                for (int j = 0; j < k; ++j) {
                    const leyline_directive& d = dirs[size_t(j)];
                    if (pos != d.span_start + delta) return fail("position bookkeeping", ci);
                    for (int64_t t = 0; t < d.stub_len; ++t, ++pos)
                        if (!check_row(pos, j, t)) return fail("replacement row", ci);
                    delta += d.stub_len - (d.span_end - d.span_start);
                    const int64_t seg_end = j + 1 < k ? dirs[size_t(j + 1)].span_start : n;
                    for (int64_t r = d.span_end; r < seg_end; ++r, ++pos)
                        if (!check_row(pos, -1, r)) return fail("moved row", ci);
                }
                if (pos != new_len) return fail("new length bookkeeping", ci);
            }
    }
    std::printf("ok %d %lld %lld\n", tile_cases, static_cast<long long>(tiles_run), static_cast<long long>(gave_up));
    return 0;
}
