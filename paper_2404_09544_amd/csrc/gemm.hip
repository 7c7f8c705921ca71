// Eq. 1 Combine for GraphSAGE: out = act([self | agg] * W) computed as
// self * W[0:d_in] + agg * W[d_in:2*d_in] with two A-operand pointers, so
// the concatenation is never stored.
//
// Matrix cores: fp32 uses v_mfma_f32_16x16x4_f32 (full fp32 products),
// bf16 uses v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  A 256-thread
// workgroup computes a BM x BN tile as 2 x 2 wavefronts; each wavefront owns
// (BM/2) x (BN/2) = several 16 x 16 MFMA tiles.  K is walked in BK steps:
// the next step's global loads are issued into registers while the current
// step's LDS tiles feed the MFMAs.  LDS rows are padded so the fragment
// reads of the four 16-lane groups fall in different banks.
//
// MFMA 16x16 fragment layouts (lane l, g = l / 16):
//   f32 x4:  A[row l%16][k g],        B[k g][col l%16]
//   bf16 x32: A[row l%16][k 8g..8g+7], B[k 8g..8g+7][col l%16]
//   result:  D[row 4g + r][col l%16] in accumulator element r.
#include "common.hpp"

namespace gnnav {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <class OutT>
__device__ __forceinline__ void store_out(OutT *c, float v);
template <>
__device__ __forceinline__ void store_out<float>(float *c, float v) { *c = v; }
template <>
__device__ __forceinline__ void store_out<uint16_t>(uint16_t *c, float v) { *c = bf16_rne(v); }

// ------------------------------------------------------------------ fp32
template <int BM, int BN, class OutT>
__global__ void __launch_bounds__(256) k_combine_f32(const float *__restrict__ A0, int64_t lda0,
                                                     const float *__restrict__ A1, int64_t lda1, int64_t M,
                                                     int64_t K, const float *__restrict__ W, int64_t N,
                                                     int relu, OutT *__restrict__ C, int64_t ldc) {
    constexpr int BK = 16;
    constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
    constexpr int PA = BM + 16, PB = BN + 16;
    constexpr int A_ROWS = BM / 64;          // float4 loads per thread for A
    constexpr int B_PER = BK * BN / 256;     // scalars per thread for B
    __shared__ float As[BK][PA];
    __shared__ float Bs[BK][PB];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid >> 1, wn = wid & 1, g = lane >> 4, l16 = lane & 15;
    const int64_t m0 = (int64_t)blockIdx.x * BM, n0 = (int64_t)blockIdx.y * BN;
    const int a_row = tid >> 2, a_k = (tid & 3) * 4;
    const int b_n = tid % BN, b_k = (tid / BN) * B_PER;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t kt = (K + BK - 1) / BK;
    const int64_t tiles = 2 * kt;
    float4 ra[A_ROWS];
    float rb[B_PER];

    auto load = [&](int64_t t) {
        const bool seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
        const float *A = seg ? A1 : A0;
        const int64_t lda = seg ? lda1 : lda0;
        const float *Wk = W + (seg ? K : 0) * N;
#pragma unroll
        for (int s = 0; s < A_ROWS; ++s) {
            const int64_t row = m0 + a_row + 64 * s;
            const int64_t k = k0 + a_k;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (row < M) {
                const float *p = A + row * lda + k;
                if (k + 3 < K) {
                    v = *(const float4 *)p;
                } else {
                    if (k < K) v.x = p[0];
                    if (k + 1 < K) v.y = p[1];
                    if (k + 2 < K) v.z = p[2];
                }
            }
            ra[s] = v;
        }
        const int64_t n = n0 + b_n;
#pragma unroll
        for (int e = 0; e < B_PER; ++e) {
            const int64_t k = k0 + b_k + e;
            rb[e] = (k < K && n < N) ? Wk[k * N + n] : 0.f;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int s = 0; s < A_ROWS; ++s) {
            As[a_k + 0][a_row + 64 * s] = ra[s].x;
            As[a_k + 1][a_row + 64 * s] = ra[s].y;
            As[a_k + 2][a_row + 64 * s] = ra[s].z;
            As[a_k + 3][a_row + 64 * s] = ra[s].w;
        }
#pragma unroll
        for (int e = 0; e < B_PER; ++e) Bs[b_k + e][b_n] = rb[e];
    };

    load(0);
    stash();
    __syncthreads();
    for (int64_t t = 0; t < tiles; ++t) {
        if (t + 1 < tiles) load(t + 1);
#pragma unroll
        for (int ks = 0; ks < BK / 4; ++ks) {
            float a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = As[ks * 4 + g][wm * WM + i * 16 + l16];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = Bs[ks * 4 + g][wn * WN + j * 16 + l16];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
        if (t + 1 < tiles) {
            stash();
            __syncthreads();
        }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t row = m0 + wm * WM + i * 16 + 4 * g + r;
                const int64_t col = n0 + wn * WN + j * 16 + l16;
                if (row < M && col < N) {
                    float v = acc[i][j][r];
                    if (relu) v = fmaxf(v, 0.f);
                    store_out<OutT>(C + row * ldc + col, v);
                }
            }
}

// ------------------------------------------------------------------ bf16
template <int BM, int BN, class OutT>
__global__ void __launch_bounds__(256) k_combine_bf16(const uint16_t *__restrict__ A0, int64_t lda0,
                                                      const uint16_t *__restrict__ A1, int64_t lda1,
                                                      int64_t M, int64_t K, const uint16_t *__restrict__ W,
                                                      int64_t N, int relu, OutT *__restrict__ C,
                                                      int64_t ldc) {
    constexpr int BK = 32;
    constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
    constexpr int PK = BK + 8;                // padded k stride (elements)
    constexpr int A_ROWS = BM / 64;           // 16-byte loads per thread for A
    constexpr int B_PER = BK * BN / 256;      // scalars per thread for B
    __shared__ __attribute__((aligned(16))) uint16_t As[BM][PK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[BN][PK];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid >> 1, wn = wid & 1, g = lane >> 4, l16 = lane & 15;
    const int64_t m0 = (int64_t)blockIdx.x * BM, n0 = (int64_t)blockIdx.y * BN;
    const int a_row = tid >> 2, a_k = (tid & 3) * 8;
    const int b_n = tid % BN, b_k = (tid / BN) * B_PER;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t kt = (K + BK - 1) / BK;
    const int64_t tiles = 2 * kt;
    uint4 ra[A_ROWS];
    uint16_t rb[B_PER];

    auto load = [&](int64_t t) {
        const bool seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
        const uint16_t *A = seg ? A1 : A0;
        const int64_t lda = seg ? lda1 : lda0;
        const uint16_t *Wk = W + (seg ? K : 0) * N;
#pragma unroll
        for (int s = 0; s < A_ROWS; ++s) {
            const int64_t row = m0 + a_row + 64 * s;
            const int64_t k = k0 + a_k;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (row < M) {
                const uint16_t *p = A + row * lda + k;
                if (k + 7 < K) {
                    v = *(const uint4 *)p;
                } else {
                    uint16_t tmp[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    for (int e = 0; e < 8; ++e)
                        if (k + e < K) tmp[e] = p[e];
                    v = make_uint4(tmp[0] | (uint32_t)tmp[1] << 16, tmp[2] | (uint32_t)tmp[3] << 16,
                                   tmp[4] | (uint32_t)tmp[5] << 16, tmp[6] | (uint32_t)tmp[7] << 16);
                }
            }
            ra[s] = v;
        }
        const int64_t n = n0 + b_n;
#pragma unroll
        for (int e = 0; e < B_PER; ++e) {
            const int64_t k = k0 + b_k + e;
            rb[e] = (k < K && n < N) ? Wk[k * N + n] : (uint16_t)0;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int s = 0; s < A_ROWS; ++s) *(uint4 *)&As[a_row + 64 * s][a_k] = ra[s];
#pragma unroll
        for (int e = 0; e < B_PER; ++e) Bs[b_n][b_k + e] = rb[e];
    };

    load(0);
    stash();
    __syncthreads();
    for (int64_t t = 0; t < tiles; ++t) {
        if (t + 1 < tiles) load(t + 1);
        bf16x8 a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = *(const bf16x8 *)&As[wm * WM + i * 16 + l16][8 * g];
#pragma unroll
        for (int j = 0; j < TN; ++j) b[j] = *(const bf16x8 *)&Bs[wn * WN + j * 16 + l16][8 * g];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        __syncthreads();
        if (t + 1 < tiles) {
            stash();
            __syncthreads();
        }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t row = m0 + wm * WM + i * 16 + 4 * g + r;
                const int64_t col = n0 + wn * WN + j * 16 + l16;
                if (row < M && col < N) {
                    float v = acc[i][j][r];
                    if (relu) v = fmaxf(v, 0.f);
                    store_out<OutT>(C + row * ldc + col, v);
                }
            }
}

template <int BN>
static void launch_combine_bn(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m,
                              int64_t d_in, const void *w, int64_t d_out, bool bf16, bool relu,
                              bool out_bf16, void *out, int64_t ld_out, hipStream_t s, const char *label) {
    constexpr int BM = 64;
    const dim3 grid((unsigned)((m + BM - 1) / BM), (unsigned)((d_out + BN - 1) / BN));
    KernelTimer t(label, s);
    if (!bf16) {
        if (out_bf16) fail(GNNAV_E_INVALID, "bf16 output needs bf16 operands");
        hipLaunchKernelGGL((k_combine_f32<BM, BN, float>), grid, dim3(256), 0, s, (const float *)self, ld_self,
                           (const float *)agg, ld_agg, m, d_in, (const float *)w, d_out, (int)relu,
                           (float *)out, ld_out);
    } else if (out_bf16) {
        hipLaunchKernelGGL((k_combine_bf16<BM, BN, uint16_t>), grid, dim3(256), 0, s, (const uint16_t *)self,
                           ld_self, (const uint16_t *)agg, ld_agg, m, d_in, (const uint16_t *)w, d_out,
                           (int)relu, (uint16_t *)out, ld_out);
    } else {
        hipLaunchKernelGGL((k_combine_bf16<BM, BN, float>), grid, dim3(256), 0, s, (const uint16_t *)self,
                           ld_self, (const uint16_t *)agg, ld_agg, m, d_in, (const uint16_t *)w, d_out,
                           (int)relu, (float *)out, ld_out);
    }
    GNNAV_HIP(hipGetLastError());
}

void launch_combine(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m, int64_t d_in,
                    const void *w, int64_t d_out, bool bf16, bool relu, bool out_bf16, void *out,
                    int64_t ld_out, hipStream_t s, const char *label) {
    if (m <= 0) return;
    if (d_out <= 64)
        launch_combine_bn<64>(self, ld_self, agg, ld_agg, m, d_in, w, d_out, bf16, relu, out_bf16, out, ld_out, s,
                              label);
    else
        launch_combine_bn<128>(self, ld_self, agg, ld_agg, m, d_in, w, d_out, bf16, relu, out_bf16, out, ld_out,
                               s, label);
}

}  // namespace gnnav
