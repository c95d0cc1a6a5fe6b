/* Prints the size and field offsets of the C ABI's structs, compiled as strict C99 from
 * include/leyline.h alone; tests/test_abi_layout.py compares them with the Python binding's
 * ctypes structures and checks the declared prototypes link against the library. */
#include <stddef.h>
#include <stdio.h>

#include "leyline.h"

#define F(T, f) printf("%s.%s %lu\n", #T, #f, (unsigned long)offsetof(T, f))
#define S(T) printf("%s %lu\n", #T, (unsigned long)sizeof(T))

int main(void) {
    S(leyline_plane);
    F(leyline_plane, base); F(leyline_plane, layer_stride); F(leyline_plane, token_stride);
    F(leyline_plane, page_stride); F(leyline_plane, row_elems); F(leyline_plane, n_heads);
    F(leyline_plane, head_stride); F(leyline_plane, rot_offset); F(leyline_plane, rot_dim);
    F(leyline_plane, rope_style); F(leyline_plane, rope_base); F(leyline_plane, inv_freq);
    S(leyline_cache);
    F(leyline_cache, dtype); F(leyline_cache, n_layers); F(leyline_cache, n_planes);
    F(leyline_cache, page_size); F(leyline_cache, capacity); F(leyline_cache, planes);
    S(leyline_directive);
    F(leyline_directive, seq); F(leyline_directive, mode); F(leyline_directive, span_start);
    F(leyline_directive, span_end); F(leyline_directive, stub_len); F(leyline_directive, stub);
    /* every entry point, taken by address so that linking checks the declarations */
    {
        typedef void (*fn_t)(void);
        const fn_t fns[] = {
            (fn_t)leyline_strerror, (fn_t)leyline_abi_version, (fn_t)leyline_pair_bits,
            (fn_t)leyline_last_hip_error,
            (fn_t)leyline_contig_query, (fn_t)leyline_splice_contig, (fn_t)leyline_splice_contig_noalloc,
            (fn_t)leyline_paged_query,
            (fn_t)leyline_paged_plan, (fn_t)leyline_splice_paged, (fn_t)leyline_rotate_delta,
        };
        size_t i, n = sizeof(fns) / sizeof(fns[0]);
        for (i = 0; i < n; ++i)
            if (!fns[i]) return 1;
        printf("entry_points %lu\n", (unsigned long)n);
    }
    printf("abi_version %d %d\n", LEYLINE_ABI_VERSION, leyline_abi_version());
    printf("strerror_overlap %s\n", leyline_strerror(LEYLINE_E_OVERLAP));
    printf("scratch_bytes %d\n", LEYLINE_SCRATCH_BYTES);
    return 0;
}
