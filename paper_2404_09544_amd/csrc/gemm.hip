// Eq. 1 Combine for GraphSAGE: out = act([self | agg] * W) computed as
// self * W[0:d_in] + agg * W[d_in:2*d_in] with two A-operand pointers, so
// the concatenation is never stored.
//
// Matrix cores: fp32 uses v_mfma_f32_16x16x4_f32 (full fp32 products),
// bf16 uses v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
//
// Main kernel (enough output tiles to fill the chip): a 256-thread
// workgroup owns a BM x BN output tile as WM x WN wavefronts, each holding
// (BM/WM) x (BN/WN) in 16 x 16 MFMA accumulators.  K is walked in BK steps
// through two LDS buffers: the next step's global loads are issued into
// registers before the current step's MFMAs and stored into the other buffer
// afterwards, so there is one barrier per step.
//
// Skinny kernel (few output rows, e.g. the last layer over the seeds): a
// workgroup owns 16 x 64 outputs; its four wavefronts take interleaved
// 16- or 32-wide K blocks straight from global memory into MFMA fragments
// and add their partial tiles in LDS in a fixed order (deterministic).
//
// MFMA 16x16 fragment layouts (lane l, g = l / 16):
//   f32 x4:   A[row l%16][k g],         B[k g][col l%16]
//   bf16 x32: A[row l%16][k 8g..8g+7],  B[k 8g..8g+7][col l%16]
//   result:   D[row 4g + r][col l%16] in accumulator element r.
// Only the pairing of A's and B's k index inside one instruction matters,
// so the loaders may assign k to (g, element) in any way that is the same
// for both operands.
#include <cstdlib>
#include <mutex>

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

template <int TM, int TN, class OutT>
__device__ __forceinline__ void write_tile(const f32x4 (&acc)[TM][TN], int64_t r0, int64_t c0, int64_t M,
                                           int64_t N, int relu, OutT *C, int64_t ldc, int g, int l16) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t row = r0 + i * 16 + 4 * g + r;
                const int64_t col = c0 + j * 16 + l16;
                if (row < M && col < N) {
                    float v = acc[i][j][r];
                    if (relu) v = fmaxf(v, 0.f);
                    store_out<OutT>(C + row * ldc + col, v);
                }
            }
}

// Workgroups are dispatched round-robin over the 8 XCDs (id % 8), each with
// its own L2.  Tiles are numbered so that the column tiles of one row band
// land on the same XCD back to back: the band's A rows are then fetched
// from HBM once and re-read from that XCD's L2.  The grid is padded to a
// multiple of 8 * ncol; padding workgroups map past the last row band.
__device__ __forceinline__ void tile_of(int64_t ncol, int64_t &tile_r, int64_t &tile_c) {
    const int64_t L = blockIdx.x, xcd = L & 7, j = L >> 3;
    tile_r = (j / ncol) * 8 + xcd;
    tile_c = j % ncol;
}

// ------------------------------------------------------------ fp32 main
// Both operands are staged as 16-byte chunks along k: A rows as stored, and
// B from WT, the weights transposed to [N][2K] once per call.  A lane's
// chunk holds four consecutive k, and MFMA q of a sub-step takes element q
// of every lane's chunk, so one 16-byte LDS read per operand feeds four
// MFMAs.  LDS slots are XOR-swizzled within each row so that both the
// chunk stores and the fragment reads are free of bank conflicts.
template <int CH>
__device__ __forceinline__ int swz(int r, int kc) {
    return r * CH + (kc ^ (CH == 4 ? ((r >> 1) & 3) : (r & 7)));
}

template <int BM, int BN, int WM, int WN, int BK>
__global__ void __launch_bounds__(256) k_combine_f32(const float *__restrict__ A0, int64_t lda0,
                                                     const float *__restrict__ A1, int64_t lda1, int64_t M,
                                                     const int32_t *__restrict__ m_dev, int64_t K,
                                                     const float *__restrict__ WT, int64_t ldb, int bvec, int nseg,
                                                     int64_t N, int relu, float *__restrict__ C, int64_t ldc) {
    constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
    constexpr int CH = BK / 4;                    // chunks per row and step
    constexpr int A_CH = BM * CH, B_CH = BN * CH;
    constexpr int A_LD = (A_CH + 255) / 256, B_LD = (B_CH + 255) / 256;
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1 && (BK == 16 || BK == 32), "tile shape");
    __shared__ f32x4 As[2][A_CH];
    __shared__ f32x4 Bs[2][B_CH];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN, g = lane >> 4, l16 = lane & 15;
    if (m_dev) M = *m_dev;
    int64_t tile_r, tile_c;
    tile_of((N + BN - 1) / BN, tile_r, tile_c);
    const int64_t m0 = tile_r * BM, n0 = tile_c * BN;
    if (m0 >= M) return;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t kt = (K + BK - 1) / BK;
    const int64_t tiles = nseg * kt;
    f32x4 ra[A_LD], rb[B_LD];

    auto chunk = [&](const float *p, int64_t k, bool vec) {
        f32x4 v = {0.f, 0.f, 0.f, 0.f};
        if (vec && k + 3 < K) {
            v = *(const f32x4 *)p;
        } else if (k + 3 < K) {
            v.x = p[0];
            v.y = p[1];
            v.z = p[2];
            v.w = p[3];
        } else {
            if (k < K) v.x = p[0];
            if (k + 1 < K) v.y = p[1];
            if (k + 2 < K) v.z = p[2];
        }
        return v;
    };
    auto load = [&](int64_t t) {
        const bool seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
        const float *A = seg ? A1 : A0;
        const int64_t lda = seg ? lda1 : lda0;
#pragma unroll
        for (int s = 0; s < A_LD; ++s) {
            const int c = tid + 256 * s;
            const int64_t row = m0 + c / CH, k = k0 + (c % CH) * 4;
            ra[s] = (c < A_CH && row < M) ? chunk(A + row * lda + k, k, true) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int s = 0; s < B_LD; ++s) {
            const int c = tid + 256 * s;
            const int64_t n = n0 + c / CH, k = k0 + (c % CH) * 4;
            rb[s] = (c < B_CH && n < N) ? chunk(WT + n * ldb + (seg ? K : 0) + k, k, bvec) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int s = 0; s < A_LD; ++s) {
            const int c = tid + 256 * s;
            if (c < A_CH) As[buf][swz<CH>(c / CH, c % CH)] = ra[s];
        }
#pragma unroll
        for (int s = 0; s < B_LD; ++s) {
            const int c = tid + 256 * s;
            if (c < B_CH) Bs[buf][swz<CH>(c / CH, c % CH)] = rb[s];
        }
    };
    // kvalid: k values of this step inside [0, K); sub-steps past them are skipped
    auto compute = [&](int buf, int64_t kvalid) {
#pragma unroll
        for (int sub = 0; sub < CH / 4; ++sub) {
            if (sub * 16 >= kvalid) break;        // uniform across the workgroup
            f32x4 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = As[buf][swz<CH>(wm * WTM + i * 16 + l16, sub * 4 + g)];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = Bs[buf][swz<CH>(wn * WTN + j * 16 + l16, sub * 4 + g)];
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
        }
    };

    load(0);
    stash(0);
    __syncthreads();
    for (int64_t t = 0; t < tiles; ++t) {
        const int buf = (int)(t & 1);
        if (t + 1 < tiles) load(t + 1);
        compute(buf, K - (t >= kt ? t - kt : t) * BK);
        if (t + 1 < tiles) stash(buf ^ 1);
        __syncthreads();
    }
    write_tile<TM, TN, float>(acc, m0 + wm * WTM, n0 + wn * WTN, M, N, relu, C, ldc, g, l16);
}

// ---------------------------------------------- fp32 main, W as stored
// Reads W row-major and stages A transposed (k-major) in LDS, one float per
// lane and k step.  Measured faster than the chunked kernel above when there
// are many row tiles over a short K (e.g. d_in = 100 over 10^5 rows).
template <int BM, int BN, int WM, int WN, int BK, class OutT>
__global__ void __launch_bounds__(256) k_combine_f32_wrow(const float *__restrict__ A0, int64_t lda0,
                                                     const float *__restrict__ A1, int64_t lda1, int64_t M,
                                                     const int32_t *__restrict__ m_dev, int64_t K,
                                                     const float *__restrict__ W, int64_t N, int relu, int wvec,
                                                     OutT *__restrict__ C, int64_t ldc) {
    constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
    constexpr int PA = BM + 16, PB = BN + 16;
    constexpr int A_CH = BM * BK / 4;             // float4 chunks in an A step
    constexpr int B_CH = BK * BN / 4;             // float4 chunks in a B step
    constexpr int A_LD = (A_CH + 255) / 256, B_LD = (B_CH + 255) / 256;
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1 && BK % 4 == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) float As[2][BK][PA];
    __shared__ __attribute__((aligned(16))) float Bs[2][BK][PB];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN, g = lane >> 4, l16 = lane & 15;
    if (m_dev) M = *m_dev;
    int64_t tile_r, tile_c;
    tile_of((N + BN - 1) / BN, tile_r, tile_c);
    const int64_t m0 = tile_r * BM, n0 = tile_c * BN;
    if (m0 >= M) return;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t kt = (K + BK - 1) / BK;
    const int64_t tiles = 2 * kt;
    float4 ra[A_LD], rb[B_LD];

    auto load = [&](int64_t t) {
        const bool seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
        const float *A = seg ? A1 : A0;
        const int64_t lda = seg ? lda1 : lda0;
        const float *Wk = W + (seg ? K : 0) * N;
#pragma unroll
        for (int s = 0; s < A_LD; ++s) {
            const int c = tid + 256 * s;
            const int r = c / (BK / 4), kq = (c % (BK / 4)) * 4;
            const int64_t row = m0 + r, k = k0 + kq;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c < A_CH && row < M) {
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
#pragma unroll
        for (int s = 0; s < B_LD; ++s) {
            const int c = tid + 256 * s;
            const int kr = c / (BN / 4), nq = (c % (BN / 4)) * 4;
            const int64_t kk = k0 + kr, n = n0 + nq;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c < B_CH && kk < K) {
                const float *q = Wk + kk * N + n;
                if (wvec && n + 3 < N) {
                    v = *(const float4 *)q;
                } else {
                    if (n < N) v.x = q[0];
                    if (n + 1 < N) v.y = q[1];
                    if (n + 2 < N) v.z = q[2];
                    if (n + 3 < N) v.w = q[3];
                }
            }
            rb[s] = v;
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int s = 0; s < A_LD; ++s) {
            const int c = tid + 256 * s;
            if (c < A_CH) {
                const int r = c / (BK / 4), kq = (c % (BK / 4)) * 4;
                As[buf][kq + 0][r] = ra[s].x;
                As[buf][kq + 1][r] = ra[s].y;
                As[buf][kq + 2][r] = ra[s].z;
                As[buf][kq + 3][r] = ra[s].w;
            }
        }
#pragma unroll
        for (int s = 0; s < B_LD; ++s) {
            const int c = tid + 256 * s;
            if (c < B_CH) *(float4 *)&Bs[buf][c / (BN / 4)][(c % (BN / 4)) * 4] = rb[s];
        }
    };

    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < BK / 4; ++ks) {
            float a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = As[buf][ks * 4 + g][wm * WTM + i * 16 + l16];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = Bs[buf][ks * 4 + g][wn * WTN + j * 16 + l16];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    };

    load(0);
    stash(0);
    __syncthreads();
    for (int64_t t = 0; t < tiles; ++t) {
        const int buf = (int)(t & 1);
        if (t + 1 < tiles) load(t + 1);
        compute(buf);
        if (t + 1 < tiles) stash(buf ^ 1);
        __syncthreads();
    }
    write_tile<TM, TN, OutT>(acc, m0 + wm * WTM, n0 + wn * WTN, M, N, relu, C, ldc, g, l16);
}


// ------------------------------------------------------------ bf16 main
// B comes from WT, the weights transposed to [N][2K] once per call, so both
// operands arrive as 16-byte chunks along k, the layout the bf16 MFMA
// fragment (8 consecutive k per lane) reads from LDS.
template <int BM, int BN, int WM, int WN, int BK, class OutT>
__global__ void __launch_bounds__(256) k_combine_bf16(const uint16_t *__restrict__ A0, int64_t lda0,
                                                      const uint16_t *__restrict__ A1, int64_t lda1,
                                                      int64_t M, const int32_t *__restrict__ m_dev, int64_t K,
                                                      const uint16_t *__restrict__ WT, int64_t N, int relu,
                                                      OutT *__restrict__ C, int64_t ldc) {
    constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
    constexpr int PK = BK + 8;                    // padded k stride (elements)
    constexpr int A_CH = BM * BK / 8;             // 16-byte chunks in an A step
    constexpr int A_LD = (A_CH + 255) / 256;
    constexpr int B_CH = BN * BK / 8;             // 16-byte chunks in a B step
    constexpr int B_LD = (B_CH + 255) / 256;
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1 && BK % 32 == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM][PK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN][PK];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN, g = lane >> 4, l16 = lane & 15;
    if (m_dev) M = *m_dev;
    int64_t tile_r, tile_c;
    tile_of((N + BN - 1) / BN, tile_r, tile_c);
    const int64_t m0 = tile_r * BM, n0 = tile_c * BN;
    if (m0 >= M) return;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t kt = (K + BK - 1) / BK;
    const int64_t tiles = 2 * kt;
    uint4 ra[A_LD], rb[B_LD];
    const int64_t K2 = 2 * K;

    auto load = [&](int64_t t) {
        const bool seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
        const uint16_t *A = seg ? A1 : A0;
        const int64_t lda = seg ? lda1 : lda0;
        const int64_t wk0 = (seg ? K : 0) + k0;
#pragma unroll
        for (int s = 0; s < A_LD; ++s) {
            const int c = tid + 256 * s;
            const int r = c / (BK / 8), kq = (c % (BK / 8)) * 8;
            const int64_t row = m0 + r, k = k0 + kq;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (c < A_CH && row < M) {
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
#pragma unroll
        for (int s = 0; s < B_LD; ++s) {
            const int c = tid + 256 * s;
            const int nr = c / (BK / 8), kq = (c % (BK / 8)) * 8;
            const int64_t n = n0 + nr, k = k0 + kq;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (c < B_CH && n < N) {
                const uint16_t *q = WT + n * K2 + wk0 + kq;
                if (k + 7 < K && (K & 7) == 0) {
                    v = *(const uint4 *)q;
                } else {
                    uint16_t tmp[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    for (int e = 0; e < 8; ++e)
                        if (k + e < K) tmp[e] = q[e];
                    v = make_uint4(tmp[0] | (uint32_t)tmp[1] << 16, tmp[2] | (uint32_t)tmp[3] << 16,
                                   tmp[4] | (uint32_t)tmp[5] << 16, tmp[6] | (uint32_t)tmp[7] << 16);
                }
            }
            rb[s] = v;
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int s = 0; s < A_LD; ++s) {
            const int c = tid + 256 * s;
            if (c < A_CH) *(uint4 *)&As[buf][c / (BK / 8)][(c % (BK / 8)) * 8] = ra[s];
        }
#pragma unroll
        for (int s = 0; s < B_LD; ++s) {
            const int c = tid + 256 * s;
            if (c < B_CH) *(uint4 *)&Bs[buf][c / (BK / 8)][(c % (BK / 8)) * 8] = rb[s];
        }
    };

    load(0);
    stash(0);
    __syncthreads();
    for (int64_t t = 0; t < tiles; ++t) {
        const int buf = (int)(t & 1);
        if (t + 1 < tiles) load(t + 1);
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            bf16x8 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[i] = *(const bf16x8 *)&As[buf][wm * WTM + i * 16 + l16][ks * 32 + 8 * g];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[j] = *(const bf16x8 *)&Bs[buf][wn * WTN + j * 16 + l16][ks * 32 + 8 * g];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (t + 1 < tiles) stash(buf ^ 1);
        __syncthreads();
    }
    write_tile<TM, TN, OutT>(acc, m0 + wm * WTM, n0 + wn * WTN, M, N, relu, C, ldc, g, l16);
}

// --------------------------------------------------------------- skinny
// 16 x 64 outputs per workgroup; wavefront w takes K blocks w, w+4, ... of
// both segments (KB = 16 fp32 or 32 bf16 wide); partial tiles are summed in
// LDS in wavefront order.
template <bool BF16>
struct Skinny;

template <>
struct Skinny<false> {
    static constexpr int KB = 16;
    // lane (row l16, group g) loads A[row][kb + 4g .. 4g+3]; MFMA s uses element s.
    __device__ static void block(const float *A, int64_t lda, int64_t row, bool row_ok, int64_t kb, int64_t K,
                                 const float *Wk, int64_t N, int64_t n0, int g, int l16, f32x4 (&acc)[4]) {
        float a[4];
        const int64_t k = kb + 4 * g;
        if (row_ok && k + 3 < K) {
            const float4 v = *(const float4 *)(A + row * lda + k);
            a[0] = v.x; a[1] = v.y; a[2] = v.z; a[3] = v.w;
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s) a[s] = (row_ok && k + s < K) ? A[row * lda + k + s] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + j * 16 + l16;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const float b = (n < N && k + s < K) ? Wk[(k + s) * N + n] : 0.f;
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b, acc[j], 0, 0, 0);
            }
        }
    }
};

template <>
struct Skinny<true> {
    static constexpr int KB = 32;
    // lane (row l16, group g) loads A[row][kb + 8g .. 8g+7] as one fragment.
    __device__ static void block(const uint16_t *A, int64_t lda, int64_t row, bool row_ok, int64_t kb,
                                 int64_t K, const uint16_t *Wk, int64_t N, int64_t n0, int g, int l16,
                                 f32x4 (&acc)[4]) {
        const int64_t k = kb + 8 * g;
        uint16_t av[8];
        if (row_ok && k + 7 < K) {
            const uint4 v = *(const uint4 *)(A + row * lda + k);
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                av[2 * e] = (uint16_t)(w[e] & 0xffffu);
                av[2 * e + 1] = (uint16_t)(w[e] >> 16);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) av[e] = (row_ok && k + e < K) ? A[row * lda + k + e] : (uint16_t)0;
        }
        bf16x8 a;
#pragma unroll
        for (int e = 0; e < 8; ++e) a[e] = __builtin_bit_cast(__bf16, av[e]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + j * 16 + l16;
            bf16x8 b;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint16_t x = (n < N && k + e < K) ? Wk[(k + e) * N + n] : (uint16_t)0;
                b[e] = __builtin_bit_cast(__bf16, x);
            }
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
        }
    }
};

template <bool BF16, class InT, class OutT>
__global__ void __launch_bounds__(256) k_combine_skinny(const InT *__restrict__ A0, int64_t lda0,
                                                        const InT *__restrict__ A1, int64_t lda1, int64_t M,
                                                        const int32_t *__restrict__ m_dev, int64_t K,
                                                        const InT *__restrict__ W, int64_t N, int relu,
                                                        OutT *__restrict__ C, int64_t ldc) {
    using S = Skinny<BF16>;
    __shared__ f32x4 part[4][4][64];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, g = lane >> 4, l16 = lane & 15;
    if (m_dev) M = *m_dev;
    const int64_t m0 = (int64_t)blockIdx.x * 16, n0 = (int64_t)blockIdx.y * 64;
    if (m0 >= M) return;
    const int64_t row = m0 + l16;
    const bool row_ok = row < M;
    f32x4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int64_t kblocks = (K + S::KB - 1) / S::KB;
    for (int64_t b = wid; b < 2 * kblocks; b += 4) {
        const bool seg = b >= kblocks;
        const int64_t kb = (seg ? b - kblocks : b) * S::KB;
        S::block(seg ? A1 : A0, seg ? lda1 : lda0, row, row_ok, kb, K, W + (seg ? K : 0) * N, N, n0, g, l16, acc);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) part[wid][j][lane] = acc[j];
    __syncthreads();
    if (wid == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f32x4 s = part[0][j][lane];
#pragma unroll
            for (int w = 1; w < 4; ++w) s += part[w][j][lane];
            acc[j] = s;
        }
        f32x4 t[1][4] = {{acc[0], acc[1], acc[2], acc[3]}};
        write_tile<1, 4, OutT>(t, m0, n0, M, N, relu, C, ldc, g, l16);
    }
}

// --------------------------------------------------------------- launch
// The main kernels read the weights transposed to [N][2K]; the copy is made
// before the kernel runs and lives in one process-wide device buffer.  An
// event recorded after the last kernel that reads it orders every later
// call after it, whichever stream that call uses.
template <class T>
__global__ void __launch_bounds__(256) k_transpose(const T *__restrict__ src, int64_t rows, int64_t cols,
                                                   T *__restrict__ dst) {
    const int64_t total = rows * cols;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t c = i / rows, r = i % rows;   // consecutive threads write consecutive dst
        dst[i] = src[r * cols + c];
    }
}

namespace {
struct SharedWorkspace {
    std::mutex mu;
    DevBuf buf;
    hipEvent_t last_use = nullptr;
};
SharedWorkspace g_wt;
}  // namespace

// WROW selects k_combine_f32_wrow for fp32 (no transposed copy of W).
template <int BM, int BN, int WM, int WN, int BKF, int BKH, bool WROW = false>
static void launch_main(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m,
                        const int32_t *m_dev, int64_t k, const void *w, int64_t n, bool bf16, bool relu,
                        bool out_bf16, void *out, int64_t ld_out, hipStream_t s, const char *label) {
    const int64_t nrow = (m + BM - 1) / BM, ncol = (n + BN - 1) / BN;
    const dim3 grid((unsigned)(((nrow + 7) / 8) * 8 * ncol));
    if (!bf16 && WROW) {
        const int wvec = (((uintptr_t)w & 15u) == 0) && n % 4 == 0;
        KernelTimer tk(label, s);
        hipLaunchKernelGGL((k_combine_f32_wrow<BM, BN, WM, WN, BKF, float>), grid, dim3(256), 0, s,
                           (const float *)self, ld_self, (const float *)agg, ld_agg, m, m_dev, k, (const float *)w, n,
                           (int)relu, wvec, (float *)out, ld_out);
        return;
    }
    std::lock_guard<std::mutex> lk(g_wt.mu);
    if (!g_wt.last_use) GNNAV_HIP(hipEventCreateWithFlags(&g_wt.last_use, hipEventDisableTiming));
    GNNAV_HIP(hipStreamWaitEvent(s, g_wt.last_use, 0));
    g_wt.buf.ensure((size_t)(2 * k * n) * (bf16 ? sizeof(uint16_t) : sizeof(float)), s);
    const dim3 tgrid(grid_for(2 * k * n, 256, 1024));
    if (!bf16) {
        float *wt = g_wt.buf.as<float>();
        {
            KernelTimer tt("weights_transpose", s);
            hipLaunchKernelGGL(k_transpose<float>, tgrid, dim3(256), 0, s, (const float *)w, 2 * k, n, wt);
        }
        KernelTimer tk(label, s);
        hipLaunchKernelGGL((k_combine_f32<BM, BN, WM, WN, BKF>), grid, dim3(256), 0, s, (const float *)self, ld_self,
                           (const float *)agg, ld_agg, m, m_dev, k, (const float *)wt, 2 * k, 1, 2, n, (int)relu,
                           (float *)out, ld_out);
    } else {
        uint16_t *wt = g_wt.buf.as<uint16_t>();
        {
            KernelTimer tt("weights_transpose", s);
            hipLaunchKernelGGL(k_transpose<uint16_t>, tgrid, dim3(256), 0, s, (const uint16_t *)w, 2 * k, n, wt);
        }
        KernelTimer tk(label, s);
        if (out_bf16)
            hipLaunchKernelGGL((k_combine_bf16<BM, BN, WM, WN, BKH, uint16_t>), grid, dim3(256), 0, s,
                               (const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m, m_dev, k,
                               (const uint16_t *)wt, n, (int)relu, (uint16_t *)out, ld_out);
        else
            hipLaunchKernelGGL((k_combine_bf16<BM, BN, WM, WN, BKH, float>), grid, dim3(256), 0, s,
                               (const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m, m_dev, k,
                               (const uint16_t *)wt, n, (int)relu, (float *)out, ld_out);
    }
    GNNAV_HIP(hipEventRecord(g_wt.last_use, s));
}

// Output tiles (counted as 64 x 64) below which the main kernel cannot fill
// 256 compute units.
constexpr int64_t kSkinnyTiles = 160;

struct GemmChoice {
    int bm, bn;
    void (*fn)(const void *, int64_t, const void *, int64_t, int64_t, const int32_t *, int64_t, const void *,
               int64_t, bool, bool, bool, void *, int64_t, hipStream_t, const char *);
};

// Tile shapes measured on MI355X.  fp32: the chunked kernel with 64 x 128
// tiles and 32-deep k steps (64 x 64 when the output is at most 64 wide);
// once there are enough 128 x 128 tiles to give every compute unit two, the
// W-as-stored kernel with 128 x 128 tiles.  bf16: 64 x 64 until that same
// 128 x 128 point.
static GemmChoice choose_main(int64_t m, int64_t d_out, bool bf16) {
#ifdef GNNAV_GEMM_SWEEP
    if (const char *e = getenv("GNNAV_GEMM_CFG")) {
        switch (atoi(e)) {
            case 1: return {64, 128, launch_main<64, 128, 2, 2, 16, 32>};
            case 2: return {64, 128, launch_main<64, 128, 2, 2, 32, 64>};
            case 3: return {128, 64, launch_main<128, 64, 2, 2, 32, 64>};
            case 4: return {128, 128, launch_main<128, 128, 2, 2, 16, 32>};
            case 5: return {64, 64, launch_main<64, 64, 2, 2, 16, 32>};
            case 6: return {64, 64, launch_main<64, 64, 2, 2, 32, 64>};
            case 8: return {128, 128, launch_main<128, 128, 2, 2, 32, 64>};
            case 9: return {128, 128, launch_main<128, 128, 2, 2, 16, 32, true>};
            case 10: return {64, 64, launch_main<64, 64, 2, 2, 16, 32, true>};
            default: break;
        }
    }
#endif
    const bool big = d_out > 64 && ((m + 127) / 128) * ((d_out + 127) / 128) >= 512;
    if (bf16) {
        if (big) return {128, 128, launch_main<128, 128, 2, 2, 16, 32>};
        return {64, 64, launch_main<64, 64, 2, 2, 16, 32>};
    }
    if (big) return {128, 128, launch_main<128, 128, 2, 2, 16, 32, true>};
    if (d_out <= 64) return {64, 64, launch_main<64, 64, 2, 2, 32, 32>};
    return {64, 128, launch_main<64, 128, 2, 2, 32, 32>};
}

void launch_combine(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m,
                    const int32_t *m_dev, int64_t d_in, const void *w, int64_t d_out, bool bf16, bool relu, bool out_bf16, void *out,
                    int64_t ld_out, hipStream_t s, const char *label) {
    if (m <= 0) return;
    if (!bf16 && out_bf16) fail(GNNAV_E_INVALID, "bf16 output needs bf16 operands");
    const GemmChoice ch = choose_main(m, d_out, bf16);
    const int64_t tiles64 = ((m + 63) / 64) * ((d_out + 63) / 64);
    if (tiles64 < kSkinnyTiles) {
        const dim3 grid((unsigned)((m + 15) / 16), (unsigned)((d_out + 63) / 64));
        KernelTimer t(label, s);
        if (!bf16)
            hipLaunchKernelGGL((k_combine_skinny<false, float, float>), grid, dim3(256), 0, s, (const float *)self,
                               ld_self, (const float *)agg, ld_agg, m, m_dev, d_in, (const float *)w, d_out,
                               (int)relu, (float *)out, ld_out);
        else if (out_bf16)
            hipLaunchKernelGGL((k_combine_skinny<true, uint16_t, uint16_t>), grid, dim3(256), 0, s,
                               (const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m, m_dev, d_in,
                               (const uint16_t *)w, d_out, (int)relu, (uint16_t *)out, ld_out);
        else
            hipLaunchKernelGGL((k_combine_skinny<true, uint16_t, float>), grid, dim3(256), 0, s,
                               (const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m, m_dev, d_in,
                               (const uint16_t *)w, d_out, (int)relu, (float *)out, ld_out);
    } else {
        ch.fn(self, ld_self, agg, ld_agg, m, m_dev, d_in, w, d_out, bf16, relu, out_bf16, out, ld_out, s, label);
    }
    GNNAV_HIP(hipGetLastError());
}

// out[M x N] = A[M x K] * B^T with B stored [N][ldb] (row n holds column n of
// the product's right operand along k): the layout of a row-major weight
// matrix read backwards, dX = dZ * W^T.  fp32, one segment, no activation.
void launch_matmul_bt(const float *a, int64_t lda, int64_t m, const int32_t *m_dev, int64_t k, const float *b,
                      int64_t ldb, int64_t n, float *out, int64_t ld_out, hipStream_t s, const char *label) {
    if (m <= 0 || n <= 0) return;
    const int bvec = (((uintptr_t)b & 15u) == 0) && ldb % 4 == 0;
    KernelTimer t(label, s);
    if (n <= 64) {
        const int64_t nrow = (m + 63) / 64, ncol = (n + 63) / 64;
        hipLaunchKernelGGL((k_combine_f32<64, 64, 2, 2, 32>), dim3((unsigned)(((nrow + 7) / 8) * 8 * ncol)), dim3(256),
                           0, s, a, lda, a, lda, m, m_dev, k, b, ldb, bvec, 1, n, 0, out, ld_out);
    } else {
        const int64_t nrow = (m + 63) / 64, ncol = (n + 127) / 128;
        hipLaunchKernelGGL((k_combine_f32<64, 128, 2, 2, 32>), dim3((unsigned)(((nrow + 7) / 8) * 8 * ncol)), dim3(256),
                           0, s, a, lda, a, lda, m, m_dev, k, b, ldb, bvec, 1, n, 0, out, ld_out);
    }
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
