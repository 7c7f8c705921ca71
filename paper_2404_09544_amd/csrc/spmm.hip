// Eq. 1 Aggregate for GraphSAGE: mean of the sampled neighbours' rows.
//
// One group of G lanes per destination row (G = 64 for wide rows, fewer for
// narrow ones so a wavefront serves 64/G rows).  Each lane owns Q 16-byte
// column units of the row (float4 or 8 x bf16) and keeps fp32 running sums
// in registers.  The group stages up to G neighbour ids in registers (one
// per lane) and broadcasts them with lane shuffles; neighbour rows are
// summed in CSR order, four rows in flight at a time.  Rows wider than
// G*Q units are done in column slabs.
#include "common.hpp"

namespace gnnav {

template <bool BF16>
struct Unit;
template <>
struct Unit<false> {
    static constexpr int kElems = 4;
    __device__ static void add(float *acc, const uint4 &v) {
        acc[0] += __uint_as_float(v.x);
        acc[1] += __uint_as_float(v.y);
        acc[2] += __uint_as_float(v.z);
        acc[3] += __uint_as_float(v.w);
    }
    __device__ static uint4 pack(const float *a) {
        return make_uint4(__float_as_uint(a[0]), __float_as_uint(a[1]), __float_as_uint(a[2]),
                          __float_as_uint(a[3]));
    }
};
template <>
struct Unit<true> {
    static constexpr int kElems = 8;
    __device__ static void add(float *acc, const uint4 &v) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc[2 * i] += __uint_as_float(w[i] << 16);
            acc[2 * i + 1] += __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    __device__ static uint4 pack(const float *a) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = (uint32_t)bf16_rne(a[2 * i]) | ((uint32_t)bf16_rne(a[2 * i + 1]) << 16);
        return make_uint4(w[0], w[1], w[2], w[3]);
    }
};

template <bool BF16, int G, int Q>
__global__ void __launch_bounds__(256) k_spmm_mean(const int32_t *__restrict__ indptr,
                                                   const int32_t *__restrict__ indices, int64_t n_dst,
                                                   const int32_t *__restrict__ n_dst_dev,
                                                   const uint4 *__restrict__ x, int64_t x_ld16,
                                                   uint4 *__restrict__ out, int64_t out_ld16, int32_t chunks,
                                                   int32_t d) {
    using U = Unit<BF16>;
    constexpr int E = U::kElems;
    constexpr int RPW = kWave / G;
    const int lane = lane_id();
    const int sub = lane / G, c0 = lane % G;
    if (n_dst_dev) n_dst = *n_dst_dev;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t r = (((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave) * RPW + sub; r < n_dst;
         r += nwaves * RPW) {
        const int32_t b = indptr[r], e = indptr[r + 1];
        const float inv = e > b ? 1.0f / (float)(e - b) : 0.0f;
        uint4 *orow = out + r * out_ld16;
        for (int32_t slab = 0; slab < chunks; slab += G * Q) {
            float acc[Q][E];
#pragma unroll
            for (int q = 0; q < Q; ++q)
#pragma unroll
                for (int t = 0; t < E; ++t) acc[q][t] = 0.0f;
            bool live[Q];
#pragma unroll
            for (int q = 0; q < Q; ++q) live[q] = slab + c0 + q * G < chunks;
            for (int32_t p0 = b; p0 < e; p0 += G) {
                const int32_t mine = p0 + c0 < e ? indices[p0 + c0] : 0;
                const int nb = min(G, e - p0);
                int j = 0;
                for (; j + 4 <= nb; j += 4) {
                    const uint4 *s0 = x + (int64_t)__shfl(mine, j, G) * x_ld16 + slab + c0;
                    const uint4 *s1 = x + (int64_t)__shfl(mine, j + 1, G) * x_ld16 + slab + c0;
                    const uint4 *s2 = x + (int64_t)__shfl(mine, j + 2, G) * x_ld16 + slab + c0;
                    const uint4 *s3 = x + (int64_t)__shfl(mine, j + 3, G) * x_ld16 + slab + c0;
                    uint4 v[4][Q];
#pragma unroll
                    for (int q = 0; q < Q; ++q) {
                        if (live[q]) {
                            v[0][q] = s0[q * G];
                            v[1][q] = s1[q * G];
                            v[2][q] = s2[q * G];
                            v[3][q] = s3[q * G];
                        }
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u)
#pragma unroll
                        for (int q = 0; q < Q; ++q)
                            if (live[q]) U::add(acc[q], v[u][q]);
                }
                for (; j < nb; ++j) {
                    const uint4 *s0 = x + (int64_t)__shfl(mine, j, G) * x_ld16 + slab + c0;
#pragma unroll
                    for (int q = 0; q < Q; ++q)
                        if (live[q]) U::add(acc[q], s0[q * G]);
                }
            }
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                if (!live[q]) continue;
                const int32_t c = slab + c0 + q * G;
                float o[E];
#pragma unroll
                for (int t = 0; t < E; ++t) o[t] = (c * E + t < d) ? acc[q][t] * inv : 0.0f;
                orow[c] = U::pack(o);
            }
        }
    }
}

template <bool BF16>
static void launch_spmm_t(const int32_t *indptr, const int32_t *indices, int64_t n_dst,
                          const int32_t *n_dst_dev, const void *x,
                          int64_t ld_x, int64_t d, void *out, int64_t ld_out, hipStream_t s,
                          const char *label) {
    constexpr int elt = BF16 ? 2 : 4;
    const int32_t chunks = (int32_t)((d * elt + 15) / 16);
    int g = 1;
    while (g < chunks && g < kWave) g <<= 1;
    int q = (chunks + g - 1) / g;
    if (q > 4) q = 4;
    const int64_t rows_per_block = (256 / kWave) * (kWave / g);
    // Grid-stride over rows: 8192 workgroups (32 per compute unit) keep the
    // memory system busy; more only adds empty workgroups when n_dst is an
    // upper bound read from the device.
    const unsigned grid = grid_for(n_dst, rows_per_block, 8192);
    const uint4 *xx = (const uint4 *)x;
    uint4 *oo = (uint4 *)out;
    const int64_t xl = ld_x * elt / 16, ol = ld_out * elt / 16;
    KernelTimer t(label, s);
#define GNNAV_L(GV, QV)                                                                             \
    hipLaunchKernelGGL((k_spmm_mean<BF16, GV, QV>), dim3(grid), dim3(256), 0, s, indptr, indices,     \
                       n_dst, n_dst_dev, xx, xl, oo, ol, chunks, (int32_t)d)
    if (g < kWave) {
        switch (g) {
            case 1: GNNAV_L(1, 1); break;
            case 2: GNNAV_L(2, 1); break;
            case 4: GNNAV_L(4, 1); break;
            case 8: GNNAV_L(8, 1); break;
            case 16: GNNAV_L(16, 1); break;
            case 32: GNNAV_L(32, 1); break;
            default: fail(GNNAV_E_INVALID, "bad row width");
        }
    } else {
        switch (q) {
            case 1: GNNAV_L(64, 1); break;
            case 2: GNNAV_L(64, 2); break;
            case 3: GNNAV_L(64, 3); break;
            default: GNNAV_L(64, 4); break;
        }
    }
#undef GNNAV_L
    GNNAV_HIP(hipGetLastError());
}

void launch_aggregate_mean(const int32_t *indptr, const int32_t *indices, int64_t n_dst,
                           const int32_t *n_dst_dev, const void *x,
                           int64_t ld_x, int64_t d, bool bf16, void *out, int64_t ld_out, hipStream_t s,
                           const char *label) {
    if (n_dst <= 0) return;
    if (bf16)
        launch_spmm_t<true>(indptr, indices, n_dst, n_dst_dev, x, ld_x, d, out, ld_out, s, label);
    else
        launch_spmm_t<false>(indptr, indices, n_dst, n_dst_dev, x, ld_x, d, out, ld_out, s, label);
}

}  // namespace gnnav
