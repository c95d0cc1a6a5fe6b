// Host-side robustness check of the planners: random, often invalid, cache descriptors and
// directives (bad dtypes, counts, strides and alignments, unsorted, overlapping or out-of-range
// spans, null replacement pointers, huge values), half of them around a valid MLA or K/V cache
// with valid directives and one field corrupted now and then.  Every call must return a status;
// built with the host sanitizers, any out-of-bounds access or undefined behaviour aborts.
//
// Usage: plan_fuzz SEED CASES   (prints "ok <plans accepted> err <plans rejected>")
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <random>
#include <vector>
#include "plan.hpp"
using namespace leyline;
int main(int argc, char** argv) {
    std::mt19937_64 rng(argc > 1 ? std::atoi(argv[1]) : 1);
    auto uni = [&](int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); };
    auto pick = [&](std::initializer_list<int64_t> v) { return *(v.begin() + uni(0, int64_t(v.size()) - 1)); };
    const int N = argc > 2 ? std::atoi(argv[2]) : 20000;
    int ok = 0, err = 0;
    for (int it = 0; it < N; ++it) {
        leyline_cache c;
        std::memset(&c, 0, sizeof(c));
        c.dtype = int32_t(pick({0, 1, 2, -1}));
        c.n_layers = int32_t(pick({0, 1, 2, 61, -3, 1 << 20}));
        c.n_planes = int32_t(pick({0, 1, 2, 4, 5, -1}));
        c.page_size = int32_t(pick({0, 0, 1, 3, 64, -2}));
        c.capacity = pick({0, 1, 100, 40000, -5, int64_t(1) << 40});
        double inv[128];
        for (int i = 0; i < 128; ++i) inv[i] = 1.0 / (i + 1);
        for (int p = 0; p < 4; ++p) {
            leyline_plane& pl = c.planes[p];
            pl.base = reinterpret_cast<void*>(pick({0, 0x100000, 0x100008}));
            pl.row_elems = int32_t(pick({576, 256, 16, 0, -8, 7}));
            pl.token_stride = pick({576, 256, 16, 0, -1, 1 << 30});
            pl.layer_stride = pick({0, 576 * 100, 16 * 40000, -16});
            pl.page_stride = pick({0, 576 * 64, 16 * 64, -16});
            pl.n_heads = int32_t(pick({1, 2, 8, 0, -1}));
            pl.head_stride = int32_t(pick({576, 128, 64, 16, 0}));
            pl.rot_offset = int32_t(pick({0, 512, 32, 8, -8}));
            pl.rot_dim = int32_t(pick({0, 64, 128, 32, 8, 7, -2}));
            pl.rope_style = int32_t(pick({0, 1, 2}));
            pl.rope_base = double(pick({10000, 0, -1}));
            pl.inv_freq = uni(0, 3) == 0 ? inv : nullptr;
        }
        if (uni(0, 1) == 0) {   // a valid descriptor: MLA, or K and V
            const bool mla = uni(0, 1) == 0;
            c.dtype = int32_t(uni(0, 1));
            c.n_layers = int32_t(uni(1, 4));
            c.n_planes = mla ? 1 : 2;
            c.page_size = int32_t(pick({0, 1, 4, 64}));
            c.capacity = pick({2000, 40000, 100000});
            for (int p = 0; p < c.n_planes; ++p) {
                leyline_plane& pl = c.planes[p];
                pl.base = reinterpret_cast<void*>(0x100000 * (p + 1));
                pl.row_elems = mla ? 576 : 256;
                pl.token_stride = pl.row_elems;
                pl.layer_stride = c.capacity * pl.row_elems * (c.page_size ? c.page_size : 1);
                pl.page_stride = int64_t(c.page_size) * pl.row_elems;
                pl.n_heads = mla ? 1 : 2;
                pl.head_stride = mla ? 576 : 128;
                pl.rot_offset = mla ? 512 : 0;
                pl.rot_dim = (mla || p == 0) ? (mla ? 64 : 128) : 0;
                pl.rope_style = mla ? 0 : 1;
                pl.rope_base = 10000.0;
                pl.inv_freq = nullptr;
            }
        }
        const int n_dirs = int(pick({0, 1, 3, 8, 40}));
        std::vector<leyline_directive> d(size_t(std::max(1, n_dirs)));
        const int64_t n = pick({0, 1, 100, 1900, 1900, 40000, -1});
        int64_t pos = 0;
        for (int j = 0; j < n_dirs; ++j) {
            leyline_directive& x = d[size_t(j)];
            std::memset(&x, 0, sizeof(x));
            x.seq = int32_t(pick({0, 0, 0, 0, 0, 1, 2, -1}));
            x.mode = int32_t(pick({0, 0, 0, 0, 0, 0, 1, 2}));
            const bool sorted = uni(0, 10) != 0;
            x.span_start = sorted ? pos + uni(0, 50) : uni(-10, 50000);
            x.span_end = x.span_start + pick({0, 1, 5, 300, -1});
            pos = x.span_end;
            x.stub_len = pick({0, 1, 16, 300, 1, 16, 0, -1, int64_t(1) << 40});
            for (int p = 0; p < 4; ++p) x.stub[p] = reinterpret_cast<const void*>(pick({0x200000, 0x200000, 0x200000, 0, 0x200004}));
        }
        if (c.n_planes >= 1 && c.n_planes <= 2 && c.planes[0].base && uni(0, 1) == 0 && n > 0) {
            // valid directives (one field corrupted one time in ten)
            std::vector<int64_t> cuts;
            for (int j = 0; j < 2 * n_dirs; ++j) cuts.push_back(uni(0, n));
            std::sort(cuts.begin(), cuts.end());
            const int n_seq_here = 3;
            for (int j = 0; j < n_dirs; ++j) {
                leyline_directive& x = d[size_t(j)];
                std::memset(&x, 0, sizeof(x));
                x.seq = c.page_size ? int32_t(uint64_t(j) * n_seq_here / uint64_t(n_dirs)) : 0;
                x.span_start = cuts[size_t(2 * j)];
                x.span_end = std::min(cuts[size_t(2 * j + 1)], x.span_start + uni(0, 300));
                x.stub_len = uni(0, 64);
                for (int p = 0; p < 4; ++p) x.stub[p] = reinterpret_cast<const void*>(0x200000 + 0x10000 * p);
            }
            if (c.page_size && n_dirs > 0) {   // per-sequence coordinates must restart: keep seq 0 only
                for (int j = 0; j < n_dirs; ++j) d[size_t(j)].seq = 0;
            }
            if (n_dirs > 0 && uni(0, 9) == 0) {
                leyline_directive& x = d[size_t(uni(0, n_dirs - 1))];
                switch (uni(0, 4)) {
                case 0: x.span_end = x.span_start - 1; break;
                case 1: x.stub_len = -1; break;
                case 2: x.stub[0] = nullptr; x.stub_len = 3; break;
                case 3: x.mode = 1; break;
                default: x.span_start = -5; break;
                }
            }
        }
        const leyline_directive* dp = uni(0, 10) == 0 ? nullptr : d.data();
        ContigSchedule cs;
        int rc = plan_contig(&c, n, dp, n_dirs, &cs);
        (rc == 0 ? ok : err)++;
        // paged
        const int n_seqs = int(pick({0, 1, 3}));
        std::vector<int32_t> lens(size_t(std::max(1, n_seqs)));
        for (auto& l : lens) l = int32_t(pick({0, 1, 100, 40000, -1}));
        PagedPlan pp;
        rc = plan_paged(int32_t(pick({1, 3, 64, 0, -1})), n_seqs, lens.data(), dp, n_dirs, int32_t(pick({1, 2, 4})),
                        uni(0, 1) == 0, &pp);
        if (rc == 0) {
            const int32_t bts = int32_t(pick({1, 10, 1000, 70000}));
            KPlane kp[LEYLINE_MAX_PLANES];
            int np = 0;
            if (check_table_width(pp, lens.data(), bts) == 0 && describe_cache(&c, true, kp, &np) == 0) {
                PagedImage img;
                rc = build_paged_image(&c, pp, n_seqs, pp.dirs, n_dirs, bts, &img);
            }
        }
        (rc == 0 ? ok : err)++;
    }
    printf("ok %d err %d\n", ok, err);
    return 0;
}
