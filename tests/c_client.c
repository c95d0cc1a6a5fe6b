/* A C program that uses libleyline.so through include/leyline.h alone: HIP device memory from
 * hipMalloc, no torch in the process.  It reads a contiguous cache and directives from a file,
 * splices the cache on the GPU with leyline_splice_contig, and writes the new length and the
 * whole cache back out; tests/test_gpu_c_client.py compares the result with the oracle.
 *
 * Input file (little endian):
 *   int32 dtype, n_layers, n_planes, capacity, seq_len, n_dirs
 *   per plane:     int32 row_elems, n_heads, head_stride, rot_offset, rot_dim, rope_style;
 *                  float64 rope_base
 *   per directive: int64 span_start, span_end, stub_len
 *   per plane:     cache [n_layers][capacity][row_elems] in the dtype
 *   per directive, per plane: replacement [n_layers][stub_len][row_elems]
 * Output file: int64 return code, int64 new length, then every plane's cache as above.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "leyline.h"

#define CHECK_HIP(x)                                                                   \
    do {                                                                               \
        hipError_t e_ = (x);                                                           \
        if (e_ != hipSuccess) {                                                        \
            fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));            \
            return 3;                                                                  \
        }                                                                              \
    } while (0)

static int read_all(FILE* f, void* p, size_t n) { return fread(p, 1, n, f) == n ? 0 : -1; }

int main(int argc, char** argv) {
    int32_t hdr[6];
    FILE* in;
    FILE* out;
    leyline_cache cache;
    leyline_directive dirs[16];
    void* dev_planes[LEYLINE_MAX_PLANES] = {0};
    void* dev_stubs[16][LEYLINE_MAX_PLANES];
    size_t plane_bytes[LEYLINE_MAX_PLANES];
    size_t esz;
    int64_t new_len = -1, ws_bytes = 0, rc;
    int32_t n_launch = 0, n_tile = 0;
    void* ws = NULL;
    int p, j;

    if (argc != 3) {
        fprintf(stderr, "usage: %s INPUT OUTPUT\n", argv[0]);
        return 2;
    }
    in = fopen(argv[1], "rb");
    if (!in || read_all(in, hdr, sizeof(hdr))) return 2;
    memset(&cache, 0, sizeof(cache));
    memset(dirs, 0, sizeof(dirs));
    memset(dev_stubs, 0, sizeof(dev_stubs));
    cache.dtype = hdr[0];
    cache.n_layers = hdr[1];
    cache.n_planes = hdr[2];
    cache.capacity = hdr[3];
    if (cache.n_planes < 1 || cache.n_planes > LEYLINE_MAX_PLANES || hdr[5] < 0 || hdr[5] > 16) return 2;
    esz = cache.dtype == LEYLINE_BF16 ? 2 : 4;
    for (p = 0; p < cache.n_planes; ++p) {
        int32_t v[6];
        double base;
        leyline_plane* pl = &cache.planes[p];
        if (read_all(in, v, sizeof(v)) || read_all(in, &base, sizeof(base))) return 2;
        pl->row_elems = v[0];
        pl->n_heads = v[1];
        pl->head_stride = v[2];
        pl->rot_offset = v[3];
        pl->rot_dim = v[4];
        pl->rope_style = v[5];
        pl->rope_base = base;
        pl->token_stride = v[0];
        pl->layer_stride = (int64_t)v[0] * cache.capacity;
        plane_bytes[p] = (size_t)cache.n_layers * (size_t)cache.capacity * (size_t)v[0] * esz;
    }
    for (j = 0; j < hdr[5]; ++j) {
        int64_t d[3];
        if (read_all(in, d, sizeof(d))) return 2;
        dirs[j].span_start = d[0];
        dirs[j].span_end = d[1];
        dirs[j].stub_len = d[2];
        dirs[j].mode = LEYLINE_AMORTIZE;
    }
    for (p = 0; p < cache.n_planes; ++p) {
        void* host = malloc(plane_bytes[p]);
        if (!host || read_all(in, host, plane_bytes[p])) return 2;
        CHECK_HIP(hipMalloc(&dev_planes[p], plane_bytes[p]));
        CHECK_HIP(hipMemcpy(dev_planes[p], host, plane_bytes[p], hipMemcpyHostToDevice));
        cache.planes[p].base = dev_planes[p];
        free(host);
    }
    for (j = 0; j < hdr[5]; ++j) {
        for (p = 0; p < cache.n_planes; ++p) {
            size_t n = (size_t)cache.n_layers * (size_t)dirs[j].stub_len * (size_t)cache.planes[p].row_elems * esz;
            void* host;
            if (n == 0) continue;
            host = malloc(n);
            if (!host || read_all(in, host, n)) return 2;
            CHECK_HIP(hipMalloc(&dev_stubs[j][p], n));
            CHECK_HIP(hipMemcpy(dev_stubs[j][p], host, n, hipMemcpyHostToDevice));
            dirs[j].stub[p] = dev_stubs[j][p];
            free(host);
        }
    }
    fclose(in);

    rc = leyline_contig_query(&cache, hdr[4], dirs, hdr[5], &new_len, &n_launch, &n_tile, &ws_bytes);
    if (rc == LEYLINE_OK && ws_bytes > 0) CHECK_HIP(hipMalloc(&ws, (size_t)ws_bytes));
    if (rc == LEYLINE_OK) rc = leyline_splice_contig(&cache, hdr[4], dirs, hdr[5], &new_len, NULL, ws, ws_bytes, NULL);
    CHECK_HIP(hipDeviceSynchronize());
    printf("rc %d (%s) new_len %ld launches %d tile_launches %d workspace %ld\n", (int)rc,
           leyline_strerror((int)rc), (long)new_len, n_launch, n_tile, (long)ws_bytes);

    out = fopen(argv[2], "wb");
    if (!out) return 2;
    fwrite(&rc, sizeof(rc), 1, out);
    fwrite(&new_len, sizeof(new_len), 1, out);
    for (p = 0; p < cache.n_planes; ++p) {
        void* host = malloc(plane_bytes[p]);
        if (!host) return 2;
        CHECK_HIP(hipMemcpy(host, dev_planes[p], plane_bytes[p], hipMemcpyDeviceToHost));
        fwrite(host, 1, plane_bytes[p], out);
        free(host);
        CHECK_HIP(hipFree(dev_planes[p]));
    }
    fclose(out);
    for (j = 0; j < hdr[5]; ++j)
        for (p = 0; p < cache.n_planes; ++p)
            if (dev_stubs[j][p]) CHECK_HIP(hipFree(dev_stubs[j][p]));
    if (ws) CHECK_HIP(hipFree(ws));
    return 0;
}
