// The row kernels' unit layout (row_unit in kparams.hpp) checked on the host for the planes the
// planner describes: every unit t below groups * tpr names a distinct (row group, chunk) of the
// item, every later t a group past its end, every chunk index stays inside the row, and with
// packed bands every full wavefront of 64 units is all band chunks or none.  Prints one line per
// plane ("plane <i> pack <B>") and exits non-zero on the first violation.
#include <cstdio>
#include <cstdlib>
#include <set>
#include <utility>

#include "plan.hpp"

using namespace leyline;

namespace {

struct PlaneCase {
    int32_t dtype, row_elems, n_heads, head_stride, rot_offset, rot_dim, style;
};

int fail(const char* what, int i, int64_t groups, int32_t t) {
    std::printf("FAIL plane %d groups %lld t %d: %s\n", i, static_cast<long long>(groups), t, what);
    return 1;
}

}  // namespace

int main() {
    const PlaneCase cases[] = {
        {LEYLINE_BF16, 576, 1, 576, 512, 64, LEYLINE_ROPE_INTERLEAVED},    // MLA c_kv + k_pe
        {LEYLINE_F32, 576, 1, 576, 512, 64, LEYLINE_ROPE_INTERLEAVED},     // the same in fp32
        {LEYLINE_BF16, 576, 1, 576, 0, 64, LEYLINE_ROPE_INTERLEAVED},      // band first
        {LEYLINE_BF16, 576, 1, 576, 256, 64, LEYLINE_ROPE_INTERLEAVED},    // band in the middle
        {LEYLINE_BF16, 512, 1, 512, 448, 16, LEYLINE_ROPE_INTERLEAVED},    // 2-chunk band
        {LEYLINE_BF16, 1024, 8, 128, 0, 128, LEYLINE_ROPE_NEOX},           // GQA K (not packed)
        {LEYLINE_BF16, 576, 1, 576, 512, 64, LEYLINE_ROPE_NEOX},           // half-split (not packed)
        {LEYLINE_BF16, 256, 1, 256, 0, 0, LEYLINE_ROPE_INTERLEAVED},       // no band (not packed)
        {LEYLINE_BF16, 520, 1, 520, 456, 64, LEYLINE_ROPE_INTERLEAVED},    // 65-chunk row (not packed)
    };
    const int64_t group_counts[] = {1, 2, 3, 7, 8, 9, 31, 63, 64, 65, 1000, 1001};
    alignas(16) static char dummy[16];
    int i = 0;
    for (const PlaneCase& c : cases) {
        leyline_cache cache{};
        cache.dtype = c.dtype;
        cache.n_layers = 1;
        cache.n_planes = 1;
        cache.capacity = 1 << 20;
        leyline_plane& pl = cache.planes[0];
        pl.base = dummy;
        pl.layer_stride = 0;
        pl.token_stride = c.row_elems;
        pl.row_elems = c.row_elems;
        pl.n_heads = c.n_heads;
        pl.head_stride = c.head_stride;
        pl.rot_offset = c.rot_offset;
        pl.rot_dim = c.rot_dim;
        pl.rope_style = c.style;
        pl.rope_base = 10000.0;
        KPlane k[LEYLINE_MAX_PLANES];
        int n = 0;
        if (describe_cache(&cache, false, k, &n) != LEYLINE_OK) return fail("describe_cache", i, 0, 0);
        const KPlane& p = k[0];
        for (int64_t groups : group_counts) {
            std::set<std::pair<int32_t, int32_t>> seen;
            const int64_t valid = groups * p.tpr;
            for (int32_t t = 0; t < int32_t(valid + 1024); ++t) {
                int32_t g, u;
                row_unit(p, true, t, groups, g, u);
                if (u < 0 || u >= p.tpr) return fail("chunk outside the row", i, groups, t);
                if (t < valid) {
                    if (g < 0 || g >= groups) return fail("valid unit names no group of the item", i, groups, t);
                    if (!seen.insert({g, u}).second) return fail("unit named twice", i, groups, t);
                } else if (g < groups) {
                    return fail("unit past the end names a group of the item", i, groups, t);
                }
            }
            if (int64_t(seen.size()) != valid) return fail("units missing", i, groups, 0);
            if (p.pack_groups) {
                const int64_t full = (groups / p.pack_groups) * p.pack_groups * p.tpr;   // whole blocks
                for (int32_t w0 = 0; w0 < int32_t(full); w0 += 64) {
                    int band = 0;
                    for (int32_t t = w0; t < w0 + 64; ++t) {
                        int32_t g, u;
                        row_unit(p, true, t, groups, g, u);
                        band += (u >= p.rot_lo && u < p.rot_lo + p.rot_chunks) ? 1 : 0;
                    }
                    if (band != 0 && band != 64) return fail("wavefront mixes band and other chunks", i, groups, w0);
                }
            }
        }
        std::printf("plane %d pack %d\n", i, p.pack_groups);
        ++i;
    }
    return 0;
}
