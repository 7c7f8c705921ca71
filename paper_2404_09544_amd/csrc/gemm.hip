// Eq. 1 Combine for GraphSAGE: out = act([self | agg] * W) computed as
// self * W[0:d_in] + agg * W[d_in:2*d_in] with two A-operand pointers, so
// the concatenation is never stored.
//
// Matrix cores: fp32 runs on the bf16 matrix cores through a three-way
// bf16 split of both operands (k_combine_split, fp32-accurate; see there);
// the backward product dX = dZ * W^T (launch_matmul_bt) uses
// v_mfma_f32_32x32x2_f32 in the ring kernel; bf16 uses
// v_mfma_f32_32x32x16_bf16 (ring) or v_mfma_f32_16x16x32_bf16 (skinny) with
// fp32 accumulation; the skinny fp32 kernel v_mfma_f32_16x16x4_f32.
//
// Ring kernel (rows 16-byte aligned; fp32 and bf16): a 256-thread
// workgroup owns a BM x BN output tile as WM x (4 / WM) wavefronts.  Both
// operands travel as 16-byte k-chunks from global memory straight into LDS
// (global_load_lds_dwordx4) through a ring of STAGES buffers, so no
// registers hold staged data and the loads of later steps are in flight
// while the current one is multiplied.  The split kernel uses the same ring.
// bf16 output tiles leave through the idle ring as 16-byte row chunks.
// Between one and 2.5 fp32 tiles per compute unit, the tiles past the
// first 256 are split along k over two or three workgroups and summed after
// (k_tail_sum), so no unit runs two whole tiles.
//
// Skinny kernel (few output rows, e.g. the last layer over the seeds): a
// workgroup owns 16 x 16 outputs; its 8 or 16 wavefronts take interleaved
// 16- or 32-wide K blocks straight from global memory into MFMA fragments
// and add their partial tiles in LDS in a fixed order (deterministic).
//
// MFMA fragment layouts (lane l):
//   f32 16x16x4:  A[row l%16][k l/16],  B[k l/16][col l%16]
//   f32 32x32x2:  A[row l%32][k l/32],  B[k l/32][col l%32]
//   bf16 16x16x32: A[row l%16][k 8(l/16)..+7], B likewise
//   bf16 32x32x16: A[row l%32][k 8(l/32)..+7], B likewise
//   16x16 result: D[row 4(l/16) + r][col l%16] in accumulator element r
//   32x32 result: D[row 8(r/4) + 4(l/32) + r%4][col l%32] in element r
// Only the pairing of A's and B's k index inside one instruction matters,
// so the loaders may assign k to (lane group, element) in any way that is
// the same for both operands.
#include <cstdlib>
#include <mutex>
#include <type_traits>

#include "bf16split.hpp"
#include "common.hpp"
#include "dma.hpp"

namespace gnnav {

typedef float f32x4 __attribute__((ext_vector_type(4)));

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

// ------------------------------------------------------- fp32 ring kernel
typedef float f32x16 __attribute__((ext_vector_type(16)));

// C = act(sum over nseg segments of A_s * B_s^T): A_s is A0 or A1 (M rows,
// stride lda_s), B_s the N rows of B at column offset s * bseg (stride ldb).
// T is float or uint16_t (bf16 bits); a 16-byte chunk holds E = 16 /
// sizeof(T) consecutive k.  Requires 16-byte aligned A0, A1, B and strides,
// bseg a multiple of E.  Step t covers k in [kb, kb + 8E) of one segment; its
// chunk (row, c) is read whole when it starts below K (a straddling chunk
// reads the row's padding) and from the row start otherwise, then the
// elements at k >= K are zeroed in LDS by the lane that loaded them, after
// its load landed and before the barrier that publishes the step.  Rows
// past M or N load the last valid row; their results are not stored.
// fp32: MFMA x of a sub-step takes element x of every lane's chunk (four
// v_mfma_f32_32x32x2_f32 per chunk pair); bf16: the chunk is the whole
// fragment of one v_mfma_f32_32x32x16_bf16 (fp32 accumulation).  Output
// OutT: float, or bf16 rounded to nearest-even.
template <class T, class OutT, int BM, int BN, int STAGES, int WM = 2>
__global__ void __launch_bounds__(256) k_combine_ring(const T *__restrict__ A0, int64_t lda0,
                                                      const T *__restrict__ A1, int64_t lda1, int64_t M,
                                                      const int32_t *__restrict__ m_dev, int64_t K,
                                                      const T *__restrict__ B, int64_t ldb, int64_t bseg, int nseg,
                                                      int64_t N, int relu, OutT *__restrict__ C, int64_t ldc) {
    constexpr bool BF16 = sizeof(T) == 2;
    constexpr int E = 16 / (int)sizeof(T), CH = 8, BK = CH * E, WN = 4 / WM;
    constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 32, TN = WTN / 32;
    constexpr int A_CH = BM * CH, B_CH = BN * CH, ST = A_CH + B_CH;
    constexpr int A_IN = A_CH / 256, B_IN = B_CH / 256, PER = A_IN + B_IN;   // DMAs per wavefront and step
    static_assert(WM * WN == 4 && TM * 32 == WTM && TN * 32 == WTN && A_CH % 256 == 0 && B_CH % 256 == 0,
                  "tile shape");
    static_assert(STAGES >= 2 && STAGES <= 3 && (STAGES - 1) * PER < 64, "ring depth");
    __shared__ f32x4 S[STAGES * ST];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN, h = lane >> 5, lr = lane & 31;
    if (m_dev) M = *m_dev;
    int64_t tile_r, tile_c;
    tile_of((N + BN - 1) / BN, tile_r, tile_c);
    const int64_t m0 = tile_r * BM, n0 = tile_c * BN;
    if (m0 >= M) return;

    // slot s = (row, chunk) with chunk stored at (chunk ^ (row & 7)): the
    // fragment reads below then touch 8 distinct 16-byte bank groups per
    // 8 lanes.  This wavefront's DMA instruction q fills slots
    // [(wid * IN + q) * 64, + 64).
    const T *pa[2][A_IN];
    int ka[A_IN];
#pragma unroll
    for (int q = 0; q < A_IN; ++q) {
        const int sl = (wid * A_IN + q) * 64 + lane, r = sl / CH;
        const int64_t row = m0 + r < M ? m0 + r : M - 1;
        pa[0][q] = A0 + row * lda0;
        pa[1][q] = A1 + row * lda1;
        ka[q] = E * ((sl % CH) ^ (r & 7));
    }
    const T *pb[B_IN];
    int kb_[B_IN];
#pragma unroll
    for (int q = 0; q < B_IN; ++q) {
        const int sl = (wid * B_IN + q) * 64 + lane, r = sl / CH;
        const int64_t n = n0 + r < N ? n0 + r : N - 1;
        pb[q] = B + n * ldb;
        kb_[q] = E * ((sl % CH) ^ (r & 7));
    }
    const int64_t kt = (K + BK - 1) / BK, steps = nseg * kt;

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    auto issue = [&](int64_t t) {
        f32x4 *buf = S + (int)(t % STAGES) * ST;
        const int seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
#pragma unroll
        for (int q = 0; q < A_IN; ++q) {
            const int64_t k = k0 + ka[q];
            dma16(pa[seg][q] + (k < K ? k : 0), &buf[(wid * A_IN + q) * 64]);
        }
#pragma unroll
        for (int q = 0; q < B_IN; ++q) {
            const int64_t k = k0 + kb_[q];
            dma16(pb[q] + seg * bseg + (k < K ? k : 0), &buf[A_CH + (wid * B_IN + q) * 64]);
        }
    };
    auto fixup = [&](int64_t t) {
        const int64_t k0 = (t >= kt ? t - kt : t) * BK;
        if (k0 + BK <= K) return;
        T *base = (T *)(S + (int)(t % STAGES) * ST);
#pragma unroll
        for (int q = 0; q < A_IN; ++q) {
            const int64_t k = k0 + ka[q];
            T *e = base + E * ((wid * A_IN + q) * 64 + lane);
#pragma unroll
            for (int x = 0; x < E; ++x)
                if (k + x >= K) e[x] = (T)0;
        }
#pragma unroll
        for (int q = 0; q < B_IN; ++q) {
            const int64_t k = k0 + kb_[q];
            T *e = base + E * (A_CH + (wid * B_IN + q) * 64 + lane);
#pragma unroll
            for (int x = 0; x < E; ++x)
                if (k + x >= K) e[x] = (T)0;
        }
    };
    // fragment of lane (h, lr) in sub-step u: row lr of its 32-row block,
    // chunk 2u + h, so k pairs up across A and B
    auto compute = [&](int64_t t) {
        const f32x4 *buf = S + (int)(t % STAGES) * ST;
#pragma unroll
        for (int u = 0; u < CH / 2; ++u) {
            f32x4 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WTM + i * 32 + lr;
                a[i] = buf[r * CH + ((2 * u + h) ^ (r & 7))];
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wn * WTN + j * 32 + lr;
                b[j] = buf[A_CH + r * CH + ((2 * u + h) ^ (r & 7))];
            }
            if constexpr (BF16) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[i]),
                                                                            __builtin_bit_cast(bf16x8, b[j]),
                                                                            acc[i][j], 0, 0, 0);
            } else {
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int i = 0; i < TM; ++i)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][x], b[j][x], acc[i][j], 0, 0, 0);
            }
        }
    };

    // every wavefront issues exactly PER DMAs per step, so "stage t landed"
    // is "at most PER * (steps issued after t) pending"
#pragma unroll
    for (int p = 0; p < STAGES - 1; ++p)
        if (p < steps) issue(p);
    for (int64_t t = 0; t < steps; ++t) {
        if (STAGES == 3 && t + 1 < steps) wait_vm<PER>();
        else wait_vm<0>();
        fixup(t);
        lds_barrier();   // stage t visible to all; everyone is done reading stage t - 1
        if (t + STAGES - 1 < steps) issue(t + STAGES - 1);
        compute(t);
    }

    if constexpr (sizeof(OutT) == 2) {
        // bf16 out: the accumulators' 2-byte column-strided stores would
        // leave each row as 64-byte pieces; the tile goes through the (now
        // idle) ring as bf16 rows instead and leaves in 16-byte row chunks
        // (7% at 107k x 256, 13% at 400k x 256 over the direct stores)
        constexpr int LDT = BN + 8, CPR = BN / 8;
        static_assert(BM * LDT * 2 <= STAGES * ST * 16, "output tile fits the ring");
        uint16_t *tile = (uint16_t *)S;
        lds_barrier();   // every wavefront is done reading the last stage
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int rl = wm * WTM + i * 32 + 8 * (r / 4) + 4 * h + (r % 4), cl = wn * WTN + j * 32 + lr;
                    float v = acc[i][j][r];
                    if (relu) v = fmaxf(v, 0.f);
                    tile[rl * LDT + cl] = bf16_rne(v);
                }
        __syncthreads();
        const bool vec = ((reinterpret_cast<uintptr_t>(C) | (uintptr_t)(ldc * 2)) & 15) == 0;
        for (int c = tid; c < BM * CPR; c += 256) {
            const int rl = c / CPR, cc = c % CPR;
            const int64_t row = m0 + rl, col = n0 + cc * 8;
            if (row >= M || col >= N) continue;
            const uint16_t *src = tile + rl * LDT + cc * 8;
            OutT *dst = C + row * ldc + col;
            if (vec && col + 8 <= N) {
                *(uint4 *)dst = *(const uint4 *)src;
            } else {
                for (int e = 0; e < 8 && col + e < N; ++e) dst[e] = src[e];
            }
        }
    } else {
        const int64_t r0 = m0 + wm * WTM, c0 = n0 + wn * WTN;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t row = r0 + i * 32 + 8 * (r / 4) + 4 * h + (r % 4), col = c0 + j * 32 + lr;
                    if (row < M && col < N) {
                        float v = acc[i][j][r];
                        if (relu) v = fmaxf(v, 0.f);
                        store_out<OutT>(C + row * ldc + col, v);
                    }
                }
    }
}

// ------------------------------------------ fp32 through split bf16
// fp32 products on the bf16 matrix cores (bf16split.hpp): both operands as
// three bf16 parts, six part products per fp32 product accumulated in fp32,
// so the result carries fp32 rounding, not bf16 rounding.  One 32x32x16 bf16
// MFMA takes half the cycles of the eight 32x32x2 fp32 MFMAs covering the
// same 16 k, so six of them cost three eighths of the plain fp32 path.
//
// Same ring as k_combine_ring: A (fp32) arrives in 16-byte k-chunks, 32 k
// per step, swizzled chunk ^ (row & 7); B arrives already split, three
// bf16 planes [3][N][ldb], 4 chunks (32 k) per plane and row per step,
// stored [plane][row][chunk ^ ((row >> 1) & 3)] so that the fragment reads
// of 8 consecutive rows hit distinct bank groups.  A fragment of sub-step
// u (16 k) is the lane's 8 fp32 values, split in registers.
template <class OutT, int BM, int BN, int WM, int STAGES = 2>
__global__ void __launch_bounds__(256) k_combine_split(const float *__restrict__ A0, int64_t lda0,
                                                       const float *__restrict__ A1, int64_t lda1, int64_t M,
                                                       const int32_t *__restrict__ m_dev, int64_t K,
                                                       const uint16_t *__restrict__ B, int64_t ldb, int64_t pstride,
                                                       int64_t bseg, int nseg, int64_t N, int relu,
                                                       OutT *__restrict__ C, int64_t ldc, int64_t Rw,
                                                       float *__restrict__ P, int64_t ldp, int64_t pseg,
                                                       int pieces) {
    constexpr int CH = 8, BK = 32, WN = 4 / WM;
    constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 32, TN = WTN / 32;
    constexpr int A_CH = BM * CH, B_PL = BN * 4, B_CH = 3 * B_PL, ST = A_CH + B_CH;
    constexpr int A_IN = A_CH / 256, B_IN = B_CH / 256, PER = A_IN + B_IN;
    static_assert(WM * WN == 4 && TM * 32 == WTM && TN * 32 == WTN && A_CH % 256 == 0 && B_CH % 256 == 0,
                  "tile shape");
    static_assert(STAGES >= 2 && STAGES <= 3 && (STAGES - 1) * PER < 64, "ring depth");
    __shared__ f32x4 S[STAGES * ST];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN, h = lane >> 5, lr = lane & 31;
    if (m_dev) M = *m_dev;
    int64_t tile_r, tile_c;
    // Workgroups below Rw * ncol take whole tiles of the first Rw row bands
    // (XCD-aware as tile_of); the rest take one of `pieces` consecutive
    // k-step ranges each of the tail bands' tiles into partial planes
    // P[0 .. pieces) (rows from Rw * BM on) that k_tail_sum adds in order.
    const int64_t ncol = (N + BN - 1) / BN, Lb = blockIdx.x, Gw = Rw * ncol;
    int64_t piece = -1, rbase = 0;
    if (Lb < Gw) {
        const int64_t xcd = Lb & 7, j = Lb >> 3;
        tile_r = (j / ncol) * 8 + xcd;
        tile_c = j % ncol;
    } else {
        const int64_t q = Lb - Gw, tile = q / pieces;
        piece = q - tile * pieces;
        tile_r = Rw + tile / ncol;
        tile_c = tile % ncol;
        rbase = Rw * BM;
    }
    const int64_t m0 = tile_r * BM, n0 = tile_c * BN;
    if (m0 >= M) return;

    const float *pa[2][A_IN];
    int ka[A_IN];
#pragma unroll
    for (int q = 0; q < A_IN; ++q) {
        const int sl = (wid * A_IN + q) * 64 + lane, r = sl / CH;
        const int64_t row = m0 + r < M ? m0 + r : M - 1;
        pa[0][q] = A0 + row * lda0;
        pa[1][q] = A1 + row * lda1;
        ka[q] = 4 * ((sl % CH) ^ (r & 7));
    }
    const uint16_t *pb[B_IN];
#pragma unroll
    for (int q = 0; q < B_IN; ++q) {
        const int sl = (wid * B_IN + q) * 64 + lane, p = sl / B_PL, rem = sl % B_PL, r = rem / 4;
        const int64_t n = n0 + r < N ? n0 + r : N - 1;
        pb[q] = B + p * pstride + n * ldb + 8 * ((rem % 4) ^ ((r >> 1) & 3));
    }
    const int64_t kt = (K + BK - 1) / BK, all_steps = nseg * kt,
                  t_first = piece < 0 ? 0 : piece * all_steps / pieces,
                  steps = piece < 0 ? all_steps : (piece + 1) * all_steps / pieces;

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    auto issue = [&](int64_t t) {
        f32x4 *buf = S + (int)(t % STAGES) * ST;
        const int seg = t >= kt;
        const int64_t k0 = (seg ? t - kt : t) * BK;
#pragma unroll
        for (int q = 0; q < A_IN; ++q) {
            const int64_t k = k0 + ka[q];
            dma16(pa[seg][q] + (k < K ? k : 0), &buf[(wid * A_IN + q) * 64]);
        }
        // B planes are zero-padded to a multiple of 32 k per segment
#pragma unroll
        for (int q = 0; q < B_IN; ++q) dma16(pb[q] + seg * bseg + k0, &buf[A_CH + (wid * B_IN + q) * 64]);
    };
    auto fixup = [&](int64_t t) {
        const int64_t k0 = (t >= kt ? t - kt : t) * BK;
        if (k0 + BK <= K) return;
        float *base = (float *)(S + (int)(t % STAGES) * ST);
#pragma unroll
        for (int q = 0; q < A_IN; ++q) {
            const int64_t k = k0 + ka[q];
            float *e = base + 4 * ((wid * A_IN + q) * 64 + lane);
#pragma unroll
            for (int x = 0; x < 4; ++x)
                if (k + x >= K) e[x] = 0.f;
        }
    };
    auto compute = [&](int64_t t) {
        const f32x4 *buf = S + (int)(t % STAGES) * ST;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            bf16x8 a1[TM], a2[TM], a3[TM], b1[TN], b2[TN], b3[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WTM + i * 32 + lr;
                const f32x4 c0 = buf[r * CH + ((4 * u + 2 * h) ^ (r & 7))];
                const f32x4 c1 = buf[r * CH + ((4 * u + 2 * h + 1) ^ (r & 7))];
                const float x[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
                split3(x, a1[i], a2[i], a3[i]);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wn * WTN + j * 32 + lr;
                const int c = (2 * u + h) ^ ((r >> 1) & 3);
                b1[j] = __builtin_bit_cast(bf16x8, buf[A_CH + r * 4 + c]);
                b2[j] = __builtin_bit_cast(bf16x8, buf[A_CH + B_PL + r * 4 + c]);
                b3[j] = __builtin_bit_cast(bf16x8, buf[A_CH + 2 * B_PL + r * 4 + c]);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = mfma_split6(a1[i], a2[i], a3[i], b1[j], b2[j], b3[j], acc[i][j]);
        }
    };

#pragma unroll
    for (int p = 0; p < STAGES - 1; ++p)
        if (t_first + p < steps) issue(t_first + p);
    // every wavefront issues exactly PER DMAs per step, so "stage t landed"
    // is "at most PER * (steps issued after t) pending"
    for (int64_t t = t_first; t < steps; ++t) {
        if (STAGES == 3 && t + 1 < steps) wait_vm<PER>();
        else wait_vm<0>();
        fixup(t);
        lds_barrier();   // stage t visible to all; everyone is done reading stage t - 1
        if (t + STAGES - 1 < steps) issue(t + STAGES - 1);
        compute(t);
    }

    const int64_t r0 = m0 + wm * WTM, c0 = n0 + wn * WTN;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = r0 + i * 32 + 8 * (r / 4) + 4 * h + (r % 4), col = c0 + j * 32 + lr;
                if (row < M && col < N) {
                    float v = acc[i][j][r];
                    if (piece >= 0) {
                        P[piece * pseg + (row - rbase) * ldp + col] = v;
                    } else {
                        if (relu) v = fmaxf(v, 0.f);
                        store_out<OutT>(C + row * ldc + col, v);
                    }
                }
            }
}

// Tail bands of a split combine: C[r] = act(P[0][r - r0] + ... +
// P[pieces - 1][r - r0]), added in piece order, for rows r0 <= r < M (M read
// on the device when m_dev is given).  V = 4: 16-byte lanes (N, ldp, pseg
// and ldc multiples of 4, P and C 16-byte aligned).
template <int V>
__global__ void __launch_bounds__(256) k_tail_sum(const float *__restrict__ P, int64_t ldp, int64_t pseg, int pieces,
                                                  int64_t r0, int64_t M, const int32_t *__restrict__ m_dev, int64_t N,
                                                  int relu, float *__restrict__ C, int64_t ldc) {
    typedef float fv __attribute__((ext_vector_type(V)));
    if (m_dev) M = *m_dev;
    const int64_t nv = N / V, total = (M - r0) * nv;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int64_t r = i / nv, c = (i - r * nv) * V;
        fv v = *(const fv *)(P + r * ldp + c);
        for (int p = 1; p < pieces; ++p) v += *(const fv *)(P + p * pseg + r * ldp + c);
        if (relu) {
#pragma unroll
            for (int e = 0; e < V; ++e) v[e] = fmaxf(v[e], 0.f);
        }
        *(fv *)(C + (r0 + r) * ldc + c) = v;
    }
}

// W [2K][N] fp32 -> its three bf16 parts, transposed: WS[p][n][kk] over
// kk in [0, 2 KP) with each K-long segment zero-padded to KP (a multiple of
// 32), the layout k_combine_split reads.  32 x 32 tiles through LDS.
__global__ void __launch_bounds__(256) k_split_transpose(const float *__restrict__ W, int64_t K, int64_t N, int64_t KP,
                                                         uint16_t *__restrict__ WS) {
    __shared__ float tile[32][33];
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    const int64_t n0 = (int64_t)blockIdx.x * 32, kk0 = (int64_t)blockIdx.y * 32;
    const int64_t seg = kk0 / KP, k0 = kk0 - seg * KP;
#pragma unroll
    for (int r = ty; r < 32; r += 8) {
        const int64_t k = k0 + r, n = n0 + tx;
        tile[r][tx] = (k < K && n < N) ? W[(seg * K + k) * N + n] : 0.f;
    }
    __syncthreads();
    const int64_t plane = N * 2 * KP;
#pragma unroll
    for (int r = ty; r < 32; r += 8) {
        const int64_t n = n0 + r;
        if (n >= N) continue;
        uint16_t p1, p2, p3;
        split3_bits(tile[tx][r], p1, p2, p3);
        uint16_t *o = WS + n * 2 * KP + kk0 + tx;
        o[0] = p1;
        o[plane] = p2;
        o[2 * plane] = p3;
    }
}

template <bool BF16, int TN>
struct Skinny;

template <int TN>
struct Skinny<false, TN> {
    static constexpr int KB = 16;
    // lane (row l16, group g) loads A[row][kb + 4g .. 4g+3]; MFMA s uses element s.
    __device__ static void block(const float *A, int64_t lda, int64_t row, bool row_ok, int64_t kb, int64_t K,
                                 const float *Wk, int64_t N, int64_t n0, int g, int l16, f32x4 (&acc)[TN]) {
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
        for (int j = 0; j < TN; ++j) {
            const int64_t n = n0 + j * 16 + l16;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const float b = (n < N && k + s < K) ? Wk[(k + s) * N + n] : 0.f;
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b, acc[j], 0, 0, 0);
            }
        }
    }
};

template <int TN>
struct Skinny<true, TN> {
    static constexpr int KB = 32;
    // lane (row l16, group g) loads A[row][kb + 8g .. 8g+7] as one fragment.
    __device__ static void block(const uint16_t *A, int64_t lda, int64_t row, bool row_ok, int64_t kb,
                                 int64_t K, const uint16_t *Wk, int64_t N, int64_t n0, int g, int l16,
                                 f32x4 (&acc)[TN]) {
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
        for (int j = 0; j < TN; ++j) {
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

// A workgroup owns 16 x 16*TN outputs.  NW wavefronts split the K blocks of
// both segments round-robin; their partial tiles are added in LDS in
// wavefront order (deterministic).  With few output rows the kernel is
// latency-bound, so many wavefronts per tile keep more loads in flight, and
// one 16-column fragment per workgroup (TN = 1) spreads a narrow output
// over more workgroups: 1024 x 512 x 41 fp32 runs in 8 us instead of 15 us
// with TN = 4.
template <bool BF16, class InT, class OutT, int NW, int TN>
__global__ void __launch_bounds__(64 * NW) k_combine_skinny(const InT *__restrict__ A0, int64_t lda0,
                                                            const InT *__restrict__ A1, int64_t lda1, int64_t M,
                                                            const int32_t *__restrict__ m_dev, int64_t K,
                                                            const InT *__restrict__ W, int64_t N, int relu,
                                                            OutT *__restrict__ C, int64_t ldc) {
    using S = Skinny<BF16, TN>;
    __shared__ f32x4 part[NW][TN][64];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, g = lane >> 4, l16 = lane & 15;
    if (m_dev) M = *m_dev;
    const int64_t m0 = (int64_t)blockIdx.x * 16, n0 = (int64_t)blockIdx.y * 16 * TN;
    if (m0 >= M) return;
    const int64_t row = m0 + l16;
    const bool row_ok = row < M;
    f32x4 acc[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int64_t kblocks = (K + S::KB - 1) / S::KB;
    for (int64_t b = wid; b < 2 * kblocks; b += NW) {
        const bool seg = b >= kblocks;
        const int64_t kb = (seg ? b - kblocks : b) * S::KB;
        S::block(seg ? A1 : A0, seg ? lda1 : lda0, row, row_ok, kb, K, W + (seg ? K : 0) * N, N, n0, g, l16, acc);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) part[wid][j][lane] = acc[j];
    __syncthreads();
    if (wid == 0) {
        f32x4 t[1][TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            f32x4 s = part[0][j][lane];
            for (int w = 1; w < NW; ++w) s += part[w][j][lane];
            t[0][j] = s;
        }
        write_tile<1, TN, OutT>(t, m0, n0, M, N, relu, C, ldc, g, l16);
    }
}

// --------------------------------------------------------------- launch
// The ring and split kernels read the weights transposed ([N][2K] rows
// along k; for the split kernel as three bf16 planes); the copy is made
// before the kernel runs, in a process-wide workspace.  An event recorded
// after the last kernel that reads it orders every later use of it after
// that kernel, whichever stream the later call comes from.
// W [2K][N] -> WT [N][2 * KP] with each K-long segment zero-padded to KP (a
// multiple of 32 and of 128 bytes), so that every 16-byte chunk the ring
// kernel starts below K lies inside its row and every row starts on a
// 128-byte boundary.  One workgroup moves a 32 (k) x 32 (n) tile through
// LDS: reads along n and writes along k are both contiguous.
template <class T>
__global__ void __launch_bounds__(256) k_transpose_pad(const T *__restrict__ W, int64_t K, int64_t N, int64_t KP,
                                                       T *__restrict__ WT) {
    __shared__ T tile[32][33];
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;          // 32 x 8 threads
    const int64_t n0 = (int64_t)blockIdx.x * 32, kk0 = (int64_t)blockIdx.y * 32;   // kk over [0, 2 KP)
    const int64_t seg = kk0 / KP, k0 = kk0 - seg * KP;                // a tile never spans segments
#pragma unroll
    for (int r = ty; r < 32; r += 8) {
        const int64_t k = k0 + r, n = n0 + tx;
        tile[r][tx] = (k < K && n < N) ? W[(seg * K + k) * N + n] : (T)0;
    }
    __syncthreads();
#pragma unroll
    for (int r = ty; r < 32; r += 8) {
        const int64_t n = n0 + r;
        if (n < N) WT[n * 2 * KP + kk0 + tx] = tile[tx][r];
    }
}

namespace {
struct SharedWorkspace {
    std::mutex mu;
    DevBuf buf;
    hipEvent_t last_use = nullptr;
};
// One workspace for all streams: combines of concurrent batches queue behind
// it (a pool of per-stream workspaces, letting two GEMMs share the chip,
// measured slower: 0.290 against 0.281 ms per step at 233k, r = 1).
SharedWorkspace g_wt;

template <int BM, int BN, class T, class OutT, int WM = 2>
void launch_ring(const T *a0, int64_t lda0, const T *a1, int64_t lda1, int64_t m, const int32_t *m_dev, int64_t k,
                 const T *b, int64_t ldb, int64_t bseg, int nseg, int64_t n, bool relu, OutT *out, int64_t ld_out,
                 hipStream_t s) {
    const int64_t nrow = (m + BM - 1) / BM, ncol = (n + BN - 1) / BN;
    const dim3 grid((unsigned)(((nrow + 7) / 8) * 8 * ncol));
    hipLaunchKernelGGL((k_combine_ring<T, OutT, BM, BN, 2, WM>), grid, dim3(256), 0, s, a0, lda0, a1, lda1, m, m_dev, k,
                       b, ldb, bseg, nseg, n, (int)relu, out, ld_out);
}
}  // namespace

// Row bands of 128 x 128 tiles taken whole when an fp32 combine splits its
// tail tiles along k (0: no split).  Between one and 2.5 tiles per compute
// unit the first 256 tiles (as 8-band groups) stay whole and the rest go to
// tail_pieces() workgroups each, one k-step range per workgroup, summed
// after by k_tail_sum: the busiest unit holds 1.33-1.5 tiles' work instead
// of 2.  Measured on MI355X (cold caches, 1204-deep k), no split -> two
// pieces: 17000 rows 119 -> 93 us, 20902 rows 124 -> 99 us, 28000 rows 144
// -> 138 us, 40000 rows 214 -> 175 us.  Below 128-deep segments the partial
// sums cost more than the balance gains (40000 x 74 x 130: 44 -> 48 us).
static int64_t tail_split_bands(int64_t m, int64_t n, int64_t k) {
    const int64_t nrow = (m + 127) / 128, ncol = (n + 127) / 128, tiles = nrow * ncol, w8 = 256 / ncol / 8 * 8;
    if (k < 128 || tiles <= 256 || tiles > 640 || w8 < 8 || w8 >= nrow) return 0;
    return w8;
}

// k-pieces per tail tile: three while the pieces fit the compute units
// about once more (the busiest unit then holds 1 + 1/3 tiles), two beyond.
// Measured at 1204-deep k (us, two -> three pieces, cold caches): 17000
// rows 103 -> 101, 20902 rows 117 -> 113, 26600 rows 154 -> 138.
static int tail_pieces(int64_t tail_tiles) { return tail_tiles <= 192 ? 3 : 2; }

// fp32: the weights are split into three bf16 parts and transposed, then
// k_combine_split runs; bf16: the weights are transposed and padded, then
// the ring kernel runs.
template <int BM, int BN>
static void launch_main(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m,
                        const int32_t *m_dev, int64_t k, const void *w, int64_t n, bool bf16, bool relu,
                        bool out_bf16, void *out, int64_t ld_out, hipStream_t s, const char *label) {
    std::lock_guard<std::mutex> lk(g_wt.mu);
    if (!g_wt.last_use) GNNAV_HIP(hipEventCreateWithFlags(&g_wt.last_use, hipEventDisableTiming));
    GNNAV_HIP(hipStreamWaitEvent(s, g_wt.last_use, 0));
    const int64_t kp = bf16 ? (k + 63) / 64 * 64 : (k + 31) / 32 * 32;
    const int64_t nrow = (m + BM - 1) / BM, ncol = (n + BN - 1) / BN, nrow8 = (nrow + 7) / 8 * 8;
    const int64_t split_bands = !bf16 && BM == 128 ? tail_split_bands(m, n, k) : 0;
    const int64_t rw = split_bands > 0 ? split_bands : nrow8;
    const int64_t tail_rows = rw < nrow ? m - rw * BM : 0;
    const int pieces = tail_rows > 0 ? tail_pieces((nrow - rw) * ncol) : 1;
    const size_t wt_bytes = (size_t)(2 * kp * n * (bf16 ? 2 : 6)), part_off = (wt_bytes + 255) / 256 * 256;
    g_wt.buf.ensure(part_off + (size_t)(pieces * tail_rows * n) * sizeof(float), s);
    const dim3 tgrid((unsigned)((n + 31) / 32), (unsigned)(2 * kp / 32));
    {
        KernelTimer tt("weights_transpose", s);
        if (!bf16)
            hipLaunchKernelGGL(k_split_transpose, tgrid, dim3(256), 0, s, (const float *)w, k, n, kp,
                               g_wt.buf.as<uint16_t>());
        else
            hipLaunchKernelGGL(k_transpose_pad<uint16_t>, tgrid, dim3(256), 0, s, (const uint16_t *)w, k, n, kp,
                               g_wt.buf.as<uint16_t>());
    }
    KernelTimer tk(label, s);
    if (!bf16) {
        const dim3 grid((unsigned)(rw * ncol + pieces * (nrow8 > rw ? nrow - rw : 0) * ncol));
        float *part = (float *)((char *)g_wt.buf.p + part_off);
        // 128 x 128 tiles as 4 x 1 wavefronts: each splits only its own 32
        // rows of A (2 x 2 split every row twice); measured 2-6% faster
        constexpr int WM = BM == 128 ? 4 : 2;
        hipLaunchKernelGGL((k_combine_split<float, BM, BN, WM>), grid, dim3(256), 0, s, (const float *)self, ld_self,
                           (const float *)agg, ld_agg, m, m_dev, k, g_wt.buf.as<uint16_t>(), 2 * kp, n * 2 * kp, kp, 2,
                           n, (int)relu, (float *)out, ld_out, rw, part, n, tail_rows * n, pieces);
        if (tail_rows > 0) {
            if (n % 4 == 0 && ld_out % 4 == 0 && ((uintptr_t)out & 15u) == 0)
                hipLaunchKernelGGL(k_tail_sum<4>, dim3(grid_for(tail_rows * n / 4, 256 * 2, 1024)), dim3(256), 0, s,
                                   part, n, tail_rows * n, pieces, rw * BM, m, m_dev, n, (int)relu, (float *)out,
                                   ld_out);
            else
                hipLaunchKernelGGL(k_tail_sum<1>, dim3(grid_for(tail_rows * n, 256 * 8, 1024)), dim3(256), 0, s,
                                   part, n, tail_rows * n, pieces, rw * BM, m, m_dev, n, (int)relu, (float *)out,
                                   ld_out);
        }
    } else if (out_bf16) {
        launch_ring<BM, BN, uint16_t, uint16_t>((const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m,
                                                m_dev, k, g_wt.buf.as<uint16_t>(), 2 * kp, kp, 2, n, relu,
                                                (uint16_t *)out, ld_out, s);
    } else {
        launch_ring<BM, BN, uint16_t, float>((const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m,
                                             m_dev, k, g_wt.buf.as<uint16_t>(), 2 * kp, kp, 2, n, relu,
                                             (float *)out, ld_out, s);
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

// Outputs of the most loaded compute unit when the tiles are dealt out
// evenly over the 256 compute units: the launch's critical path.
static int64_t busiest_cu_outputs(int64_t m, int64_t n, int64_t bm, int64_t bn) {
    const int64_t tiles = ((m + bm - 1) / bm) * ((n + bn - 1) / bn);
    return (tiles + 255) / 256 * bm * bn;
}

// Busiest compute unit's outputs under the tail split: one whole tile plus
// its share of the tail tiles' k-pieces.
static int64_t busiest_cu_outputs_tail(int64_t m, int64_t n) {
    const int64_t tiles = ((m + 127) / 128) * ((n + 127) / 128), tail = tiles - 256;
    const int p = tail_pieces(tail);
    return 128 * 128 * (p + (p * tail + 255) / 256) / p;
}

// Tile shapes measured on MI355X.  fp32 (split kernel): 128 x 128 or
// 64 x 64, whichever loads the busiest compute unit less, counting a 64 x 64
// output as 1/0.7 of its size (its per-output rate measured ~0.7 of the
// larger tile's) and 128 x 128 with the tail split where it applies: e.g.
// 17000 and 20902 x 1204 x 256 take 128 x 128, 6915 x 256 x 256 and 40000 x
// 74 x 130 take 64 x 64.  bf16 (ring kernel): 128 x 64
// tiles (64 x 64 for outputs at most 64 wide), 128 x 128 once there are
// enough of those to give every compute unit two.
static GemmChoice choose_main(int64_t m, int64_t d_in, int64_t d_out, bool bf16) {
    if (bf16) {
        const bool big = d_out > 64 && ((m + 127) / 128) * ((d_out + 127) / 128) >= 512;
        if (big) return {128, 128, launch_main<128, 128>};
        if (d_out <= 64) return {64, 64, launch_main<64, 64>};
        return {128, 64, launch_main<128, 64>};
    }
    const int64_t b128 = tail_split_bands(m, d_out, d_in) > 0 ? busiest_cu_outputs_tail(m, d_out)
                                                               : busiest_cu_outputs(m, d_out, 128, 128);
    if (d_out > 64 && 7 * b128 <= 10 * busiest_cu_outputs(m, d_out, 64, 64)) return {128, 128, launch_main<128, 128>};
    return {64, 64, launch_main<64, 64>};
}

int combine_kernel_kind(int64_t m, int64_t d_out, bool bf16) {
    const int64_t tiles64 = ((m + 63) / 64) * ((d_out + 63) / 64);
    if (tiles64 < kSkinnyTiles) return GNNAV_COMBINE_SKINNY;
    return bf16 ? GNNAV_COMBINE_RING : GNNAV_COMBINE_SPLIT;
}

void launch_combine(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m,
                    const int32_t *m_dev, int64_t d_in, const void *w, int64_t d_out, bool bf16, bool relu, bool out_bf16, void *out,
                    int64_t ld_out, hipStream_t s, const char *label) {
    if (m <= 0) return;
    if (!bf16 && out_bf16) fail(GNNAV_E_INVALID, "bf16 output needs bf16 operands");
    if (combine_kernel_kind(m, d_out, bf16) == GNNAV_COMBINE_SKINNY) {
        // one 16 x 16 output fragment per workgroup; 16 wavefronts split K
        // while that leaves at most 512 workgroups, 8 beyond (measured)
        const dim3 grid((unsigned)((m + 15) / 16), (unsigned)((d_out + 15) / 16));
        KernelTimer t(label, s);
        auto run = [&](auto nw) {
            constexpr int NW = decltype(nw)::value;
            if (!bf16)
                hipLaunchKernelGGL((k_combine_skinny<false, float, float, NW, 1>), grid, dim3(64 * NW), 0, s,
                                   (const float *)self, ld_self, (const float *)agg, ld_agg, m, m_dev, d_in,
                                   (const float *)w, d_out, (int)relu, (float *)out, ld_out);
            else if (out_bf16)
                hipLaunchKernelGGL((k_combine_skinny<true, uint16_t, uint16_t, NW, 1>), grid, dim3(64 * NW), 0, s,
                                   (const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m, m_dev, d_in,
                                   (const uint16_t *)w, d_out, (int)relu, (uint16_t *)out, ld_out);
            else
                hipLaunchKernelGGL((k_combine_skinny<true, uint16_t, float, NW, 1>), grid, dim3(64 * NW), 0, s,
                                   (const uint16_t *)self, ld_self, (const uint16_t *)agg, ld_agg, m, m_dev, d_in,
                                   (const uint16_t *)w, d_out, (int)relu, (float *)out, ld_out);
        };
        if ((int64_t)grid.x * grid.y <= 512)
            run(std::integral_constant<int, 16>{});
        else
            run(std::integral_constant<int, 8>{});
    } else {
        const GemmChoice ch = choose_main(m, d_in, d_out, bf16);
        ch.fn(self, ld_self, agg, ld_agg, m, m_dev, d_in, w, d_out, bf16, relu, out_bf16, out, ld_out, s, label);
    }
    GNNAV_HIP(hipGetLastError());
}

// out[M x N] = A[M x K] * B^T with B stored [N][ldb] (row n holds column n of
// the product's right operand along k): the layout of a row-major weight
// matrix read backwards, dX = dZ * W^T.  fp32, one segment, no activation.
// Rows [n][k] at stride ldb -> [n][k4] (k4 = k rounded up to 4), zero padded,
// for operands whose rows are not 16-byte aligned.
__global__ void __launch_bounds__(256) k_pad_rows(const float *__restrict__ b, int64_t ldb, int64_t n, int64_t k,
                                                  int64_t k4, float *__restrict__ out) {
    const int64_t total = n * k4, stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t r = i / k4, c = i - r * k4;
        out[i] = c < k ? b[r * ldb + c] : 0.f;
    }
}

void launch_matmul_bt(const float *a, int64_t lda, int64_t m, const int32_t *m_dev, int64_t k, const float *b,
                      int64_t ldb, int64_t n, float *out, int64_t ld_out, hipStream_t s, const char *label) {
    if (m <= 0 || n <= 0) return;
    if (!((((uintptr_t)a & 15u) == 0) && lda % 4 == 0))
        fail(GNNAV_E_INVALID, "matmul_bt: rows of a must be 16-byte aligned");
    auto run = [&](const float *bb, int64_t ldbb) {
        KernelTimer t(label, s);
        if (n <= 64)
            launch_ring<64, 64>(a, lda, a, lda, m, m_dev, k, bb, ldbb, 0, 1, n, false, out, ld_out, s);
        else
            launch_ring<128, 64>(a, lda, a, lda, m, m_dev, k, bb, ldbb, 0, 1, n, false, out, ld_out, s);
    };
    if ((((uintptr_t)b & 15u) == 0) && ldb % 4 == 0) {
        run(b, ldb);
    } else {
        // rows of b not 16-byte aligned (W of a layer with an odd output
        // width): a zero-padded copy in the shared weights buffer first
            std::lock_guard<std::mutex> lk(g_wt.mu);
        if (!g_wt.last_use) GNNAV_HIP(hipEventCreateWithFlags(&g_wt.last_use, hipEventDisableTiming));
        GNNAV_HIP(hipStreamWaitEvent(s, g_wt.last_use, 0));
        const int64_t k4 = (k + 3) / 4 * 4;
        g_wt.buf.ensure((size_t)(n * k4) * sizeof(float), s);
        hipLaunchKernelGGL(k_pad_rows, dim3(grid_for(n * k4, 256, 1024)), dim3(256), 0, s, b, ldb, n, k, k4,
                           g_wt.buf.as<float>());
        run(g_wt.buf.as<float>(), k4);
        GNNAV_HIP(hipEventRecord(g_wt.last_use, s));
    }
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
