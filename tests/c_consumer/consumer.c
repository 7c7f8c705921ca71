/* A plain C program that runs one sampled mini-batch through the C ABI of
 * libgnnav.so (include/gnnav.h) with no Python and no torch: build the CSR
 * and the degree-ranked cache, sample the batch (Eq. 2), gather F_L's rows
 * (the cache step of Section 3.2) and run the L-layer SAGE forward (Eq. 1).
 * Device buffers come from the HIP runtime's C API.  Test infrastructure:
 * tests/test_gpu_c_consumer.py writes the problem and checks the result
 * against the oracle.
 *
 * usage: consumer PROBLEM OUT
 * PROBLEM (little-endian): int64 n, m, d, L, n_seeds; double r;
 *   uint64 rng_seed; int32 src[m], dst[m]; float feats[n*d];
 *   int32 fanouts[L]; int32 dims[L+1]; int32 seeds[n_seeds];
 *   then for l = 1..L float W_l[2*dims[l-1]*dims[l]] (row-major).
 * The batch runs on a stream restricted to one half of the compute units
 * (gnnav_stream_create), which changes no result.
 * OUT: int64 sizes[L+1]; int64 counts[3]; float logits[sizes[0]*dims[L]].
 * Exit status 0 on success; on a failing call the status, the call and
 * gnnav_last_error() go to stderr and the status is 1. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "gnnav.h"

#define CHECK(call)                                                                                   \
    do {                                                                                              \
        gnnav_status st_ = (call);                                                                    \
        if (st_ != GNNAV_OK) {                                                                        \
            fprintf(stderr, "%s -> status %d: %s\n", #call, (int)st_, gnnav_last_error());            \
            return 1;                                                                                 \
        }                                                                                             \
    } while (0)
#define HIP(call)                                                                                     \
    do {                                                                                              \
        hipError_t e_ = (call);                                                                       \
        if (e_ != hipSuccess) {                                                                       \
            fprintf(stderr, "%s -> %s\n", #call, hipGetErrorString(e_));                              \
            return 1;                                                                                 \
        }                                                                                             \
    } while (0)

static int read_exact(FILE *f, void *dst, size_t bytes) { return fread(dst, 1, bytes, f) == bytes ? 0 : -1; }

int main(int argc, char **argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s PROBLEM OUT\n", argv[0]);
        return 2;
    }
    FILE *f = fopen(argv[1], "rb");
    if (!f) {
        fprintf(stderr, "cannot open %s\n", argv[1]);
        return 2;
    }
    int64_t hdr[5];
    double r;
    uint64_t rng_seed;
    if (read_exact(f, hdr, sizeof hdr) || read_exact(f, &r, sizeof r) || read_exact(f, &rng_seed, sizeof rng_seed))
        return 2;
    const int64_t n = hdr[0], m = hdr[1], d = hdr[2], L = hdr[3], n_seeds = hdr[4];
    if (n <= 0 || m < 0 || d <= 0 || L < 1 || L > 16 || n_seeds < 0) return 2;
    int32_t *src = malloc((size_t)(m ? m : 1) * 4), *dst = malloc((size_t)(m ? m : 1) * 4);
    float *feats = malloc((size_t)(n * d) * 4);
    int32_t fanouts[16], dims[17];
    int32_t *seeds = malloc((size_t)(n_seeds ? n_seeds : 1) * 4);
    if (!src || !dst || !feats || !seeds) return 2;
    if (read_exact(f, src, (size_t)m * 4) || read_exact(f, dst, (size_t)m * 4) ||
        read_exact(f, feats, (size_t)(n * d) * 4) || read_exact(f, fanouts, (size_t)L * 4) ||
        read_exact(f, dims, (size_t)(L + 1) * 4) || read_exact(f, seeds, (size_t)n_seeds * 4))
        return 2;
    float *w_host[16];
    for (int64_t l = 1; l <= L; ++l) {
        const size_t bytes = (size_t)(2 * dims[l - 1]) * (size_t)dims[l] * 4;
        w_host[l - 1] = malloc(bytes);
        if (!w_host[l - 1] || read_exact(f, w_host[l - 1], bytes)) return 2;
    }
    fclose(f);
    if (gnnav_abi_version() != GNNAV_ABI_VERSION) {
        fprintf(stderr, "ABI version %d, header %d\n", gnnav_abi_version(), GNNAV_ABI_VERSION);
        return 1;
    }
    /* freeing NULL handles is allowed */
    gnnav_graph_free(NULL);
    gnnav_cache_free(NULL);
    gnnav_blocks_free(NULL);
    CHECK(gnnav_stream_destroy(NULL));
    void *stream = NULL;
    CHECK(gnnav_stream_create(1, 2, &stream));

    gnnav_graph *g = NULL;
    gnnav_cache *c = NULL;
    gnnav_blocks *b = NULL;
    CHECK(gnnav_build_csr(n, m, src, dst, GNNAV_SYMMETRIZE, &g));
    CHECK(gnnav_build_cache(g, feats, d, GNNAV_F32, r, 0u, &c));
    int64_t ld = 0;
    CHECK(gnnav_cache_info(c, NULL, NULL, &ld, NULL, NULL));
    CHECK(gnnav_blocks_create(&b));

    int32_t *seeds_d = NULL;
    HIP(hipMalloc((void **)&seeds_d, (size_t)(n_seeds ? n_seeds : 1) * 4));
    HIP(hipMemcpy(seeds_d, seeds, (size_t)n_seeds * 4, hipMemcpyHostToDevice));
    CHECK(gnnav_sample(g, seeds_d, n_seeds, fanouts, (int32_t)L, rng_seed, b, stream));

    const int32_t *nodes_d = NULL;
    int64_t sizes[17];
    int32_t hops = 0;
    CHECK(gnnav_blocks_nodes(b, &nodes_d, sizes, &hops));
    if (hops != L) {
        fprintf(stderr, "blocks hold %d hops, expected %lld\n", hops, (long long)L);
        return 1;
    }
    for (int32_t h = 1; h <= hops; ++h) {
        gnnav_block_view v;
        CHECK(gnnav_blocks_hop(b, h, &v));
        if (v.n_dst != sizes[h - 1] || v.n_src != sizes[h]) {
            fprintf(stderr, "hop %d view disagrees with the node list sizes\n", h);
            return 1;
        }
    }

    float *h0 = NULL, *logits = NULL;
    int64_t *counts_d = NULL;
    HIP(hipMalloc((void **)&h0, (size_t)(sizes[L] ? sizes[L] : 1) * (size_t)ld * 4));
    HIP(hipMalloc((void **)&counts_d, 3 * sizeof(int64_t)));
    CHECK(gnnav_gather(c, nodes_d, sizes[L], h0, ld, counts_d, stream));

    float *w_dev[16];
    for (int64_t l = 1; l <= L; ++l) {
        const size_t bytes = (size_t)(2 * dims[l - 1]) * (size_t)dims[l] * 4;
        HIP(hipMalloc((void **)&w_dev[l - 1], bytes));
        HIP(hipMemcpy(w_dev[l - 1], w_host[l - 1], bytes, hipMemcpyHostToDevice));
    }
    const int64_t ld_out = dims[L];
    HIP(hipMalloc((void **)&logits, (size_t)(sizes[0] ? sizes[0] : 1) * (size_t)ld_out * 4));
    CHECK(gnnav_sage_forward(b, h0, ld, (const void *const *)w_dev, dims, (int32_t)L, GNNAV_F32, logits, ld_out,
                             stream));
    CHECK(gnnav_sync(stream));

    int64_t counts[3];
    float *out_logits = malloc((size_t)(sizes[0] ? sizes[0] : 1) * (size_t)ld_out * 4);
    if (!out_logits) return 2;
    HIP(hipMemcpy(counts, counts_d, sizeof counts, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(out_logits, logits, (size_t)sizes[0] * (size_t)ld_out * 4, hipMemcpyDeviceToHost));

    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    fwrite(sizes, sizeof(int64_t), (size_t)(L + 1), o);
    fwrite(counts, sizeof(int64_t), 3, o);
    fwrite(out_logits, 4, (size_t)sizes[0] * (size_t)ld_out, o);
    fclose(o);

    for (int64_t l = 0; l < L; ++l) {
        HIP(hipFree(w_dev[l]));
        free(w_host[l]);
    }
    HIP(hipFree(logits));
    HIP(hipFree(counts_d));
    HIP(hipFree(h0));
    HIP(hipFree(seeds_d));
    gnnav_blocks_free(b);
    gnnav_cache_free(c);
    gnnav_graph_free(g);
    CHECK(gnnav_stream_destroy(stream));
    free(out_logits);
    free(seeds);
    free(feats);
    free(dst);
    free(src);
    return 0;
}
