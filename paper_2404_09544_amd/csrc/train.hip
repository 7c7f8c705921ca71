// The training half of the iteration (the loss, backward and update steps
// of Algorithm 1), fp32:
//
//   softmax_xent   one wavefront per row of the logits: row max, sum of
//                  exponentials, the row's loss and its gradient
//                  (softmax - onehot) / n; the batch loss is summed by one
//                  workgroup in a fixed order
//   csc            the transpose of a sampled block, by a stable LSD radix
//                  sort of (source local id, destination row) pairs in edge
//                  order, so every column lists its edges in edge order;
//                  column pointers by a lower-bound search of the sorted keys
//   aggregate_t    the adjoint of the mean aggregation: for each source row j,
//                  the sum over its column of dAgg[i] / cnt_i, in column
//                  order, plus the self-term gradient, times the ReLU mask of
//                  the layer below; no floating-point atomics, so the result
//                  is the same on every run
//   wgrad          dW = [X_self | Agg]^T dZ (bf16 matrix cores through the
//                  three-way bf16 split): MFMA tiles over (input feature,
//                  output feature), the row dimension split into ranges whose
//                  partial tiles are summed in range order by the reduce
//                  kernel, which also applies W -= lr * dW
#include <algorithm>

#include "common.hpp"
#include "bf16split.hpp"
#include "dma.hpp"
#include "scan.hpp"

namespace gnnav {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ softmax-CE
__global__ void __launch_bounds__(256) k_softmax_xent(const float *__restrict__ Z, int64_t ldz, int64_t n,
                                                      const int32_t *__restrict__ n_dev, int64_t C,
                                                      const int32_t *__restrict__ nodes,
                                                      const int32_t *__restrict__ labels, float *__restrict__ dZ,
                                                      int64_t lddz, float *__restrict__ row_loss) {
    if (n_dev) n = *n_dev;
    const int lane = lane_id();
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    const float inv_n = n > 0 ? 1.0f / (float)n : 0.0f;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; i < n; i += nwaves) {
        const float *z = Z + i * ldz;
        float mx = -INFINITY;
        for (int64_t c = lane; c < C; c += kWave) mx = fmaxf(mx, z[c]);
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
        float se = 0.0f;
        for (int64_t c = lane; c < C; c += kWave) se += expf(z[c] - mx);
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) se += __shfl_xor(se, o, kWave);
        const int32_t y = labels[nodes ? nodes[i] : i];
        const bool ok = y >= 0 && y < C;
        const float inv_se = 1.0f / se;
        float *g = dZ + i * lddz;
        for (int64_t c = lane; c < C; c += kWave) {
            const float p = expf(z[c] - mx) * inv_se;
            g[c] = ok ? (p - (c == y ? 1.0f : 0.0f)) * inv_n : 0.0f;
        }
        if (lane == 0) row_loss[i] = ok ? logf(se) + mx - z[y] : NAN;
    }
}

// One workgroup: thread t sums rows t, t + 256, ... in double; the partial
// sums are combined by a fixed tree.
__global__ void __launch_bounds__(256) k_loss_mean(const float *__restrict__ row_loss, int64_t n,
                                                   const int32_t *__restrict__ n_dev, float *__restrict__ out) {
    __shared__ double part[256];
    if (n_dev) n = *n_dev;
    double s = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += 256) s += (double)row_loss[i];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = n > 0 ? (float)(part[0] / (double)n) : 0.0f;
}

void launch_softmax_xent(const float *z, int64_t ldz, int64_t n, const int32_t *n_dev, int64_t C,
                         const int32_t *nodes, const int32_t *labels, float *dz, int64_t lddz, float *row_loss,
                         float *loss, hipStream_t s) {
    if (n > 0) {
        KernelTimer t("softmax_xent", s);
        hipLaunchKernelGGL(k_softmax_xent, dim3(grid_for(n, 4, 4096)), dim3(256), 0, s, z, ldz, n, n_dev, C, nodes,
                           labels, dz, lddz, row_loss);
    }
    {
        KernelTimer t("loss_mean", s);
        hipLaunchKernelGGL(k_loss_mean, dim3(1), dim3(256), 0, s, row_loss, n, n_dev, loss);
    }
    GNNAV_HIP(hipGetLastError());
}

// ---------------------------------------------------------------- CSC
constexpr int kSortThreads = 256;
constexpr int kSortIters = 8;
constexpr int kSortTile = kSortThreads * kSortIters;   // elements per workgroup

__global__ void __launch_bounds__(256) k_edge_rows(const int32_t *__restrict__ indptr, int64_t n_dst,
                                                   const int32_t *__restrict__ n_dev, int32_t *__restrict__ rows) {
    if (n_dev) n_dst = *n_dev;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_dst; i += stride)
        for (int32_t p = indptr[i]; p < indptr[i + 1]; ++p) rows[p] = (int32_t)i;
}

// Elements of tile t: t * kSortTile + it * 256 + thread, it = 0 .. 7, so a
// workgroup meets its elements in index order, 256 at a time.
__global__ void __launch_bounds__(256) k_radix_hist(const int32_t *__restrict__ keys, const int32_t *__restrict__ n_ptr,
                                                    int shift, int32_t *__restrict__ hist, int64_t ntiles) {
    __shared__ int32_t h[256];
    const int64_t n = *n_ptr;
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int it = 0; it < kSortIters; ++it) {
        const int64_t e = base + it * kSortThreads + threadIdx.x;
        if (e < n) atomicAdd(&h[(keys[e] >> shift) & 255], 1);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

struct HistScanOp {
    const int32_t *hist;
    int32_t *offs;
    int64_t count;
    __device__ int64_t n() const { return count; }
    __device__ int32_t value(int64_t i) const { return hist[i]; }
    __device__ void emit(int64_t i, int32_t prefix, int32_t) const { offs[i] = prefix; }
    __device__ void total(int32_t) const {}
};

// Stable scatter: an element's destination is its digit's offset for this
// tile, plus the elements of the same digit earlier in the tile.  Within a
// wavefront the earlier same-digit lanes come from eight ballots (one per
// digit bit); across the four wavefronts and the eight passes, from LDS
// counters.
__global__ void __launch_bounds__(256) k_radix_scatter(const int32_t *__restrict__ keys_in,
                                                       const int32_t *__restrict__ vals_in,
                                                       const int32_t *__restrict__ n_ptr, int shift,
                                                       const int32_t *__restrict__ offs, int64_t ntiles,
                                                       int32_t *__restrict__ keys_out, int32_t *__restrict__ vals_out) {
    __shared__ int32_t run[256];
    __shared__ int32_t cnt[kSortThreads / kWave][256];
    const int64_t n = *n_ptr;
    const int lane = lane_id(), wid = threadIdx.x / kWave;
    run[threadIdx.x] = offs[(int64_t)threadIdx.x * ntiles + blockIdx.x];
    const uint64_t below = (1ull << lane) - 1ull;
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int it = 0; it < kSortIters; ++it) {
#pragma unroll
        for (int w = 0; w < kSortThreads / kWave; ++w) cnt[w][threadIdx.x] = 0;
        __syncthreads();
        const int64_t e = base + it * kSortThreads + threadIdx.x;
        const bool valid = e < n;
        const int32_t key = valid ? keys_in[e] : 0;
        const int d = (key >> shift) & 255;
        uint64_t m = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const uint64_t ones = __ballot(valid && ((d >> bit) & 1));
            m &= ((d >> bit) & 1) ? ones : ~ones;
        }
        const int rank = __popcll(m & below);
        if (valid && rank == 0) cnt[wid][d] = __popcll(m);
        __syncthreads();
        if (valid) {
            int32_t pos = run[d] + rank;
            for (int w = 0; w < wid; ++w) pos += cnt[w][d];
            keys_out[pos] = key;
            vals_out[pos] = vals_in[e];
        }
        __syncthreads();
        int32_t add = 0;
#pragma unroll
        for (int w = 0; w < kSortThreads / kWave; ++w) add += cnt[w][threadIdx.x];
        run[threadIdx.x] += add;
        __syncthreads();
    }
}

// Column pointers from the sorted keys: col_ptr[s] = the number of keys
// below s (a lower-bound search per s), for s in [0, n_src_bound].  The keys
// are local source ids, all below n_src_bound.
__global__ void __launch_bounds__(256) k_col_ptr(const int32_t *__restrict__ keys, const int32_t *__restrict__ n_ptr,
                                                 int64_t n_src_bound, int32_t *__restrict__ col_ptr) {
    const int64_t n = *n_ptr;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c <= n_src_bound; c += stride) {
        int64_t lo = 0, hi = n;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (keys[mid] < c) lo = mid + 1;
            else hi = mid;
        }
        col_ptr[c] = (int32_t)lo;
    }
}

// Sorted (source, destination row) pairs of one block and its column
// pointers.  n_edges_dev: device edge count (<= e_bound); n_src_bound sizes
// the key range; the buffers are grow-only.
void CscWorkspace::build(const int32_t *indptr, const int32_t *indices, int64_t n_dst, const int32_t *n_dst_dev,
                         const int32_t *n_edges_dev, int64_t e_bound, int64_t n_src_bound, ScanState &scan,
                         hipStream_t s, const char *label) {
    KernelTimer t(label, s);
    const int64_t eb = std::max<int64_t>(e_bound, 1);
    const int64_t ntiles = (eb + kSortTile - 1) / kSortTile;
    for (int k = 0; k < 2; ++k) {
        keys[k].ensure(eb * sizeof(int32_t), s);
        vals[k].ensure(eb * sizeof(int32_t), s);
    }
    hist.ensure(256 * ntiles * sizeof(int32_t), s);
    offs.ensure(256 * ntiles * sizeof(int32_t), s);
    col_ptr.ensure((n_src_bound + 1) * sizeof(int32_t), s);
    // pass 0 reads the block's indices directly; values are destination rows
    hipLaunchKernelGGL(k_edge_rows, dim3(grid_for(n_dst, 256, 4096)), dim3(256), 0, s, indptr, n_dst, n_dst_dev,
                       vals[1].as<int32_t>());
    int bits = 1;
    while (bits < 31 && (int64_t(1) << bits) < n_src_bound) ++bits;
    const int passes = (bits + 7) / 8;
    const int32_t *kin = indices, *vin = vals[1].as<int32_t>();
    int cur = 0;
    scan.ensure(256 * ntiles, s);
    for (int p = 0; p < passes; ++p) {
        int32_t *kout = keys[cur].as<int32_t>(), *vout = vals[cur].as<int32_t>();
        hipLaunchKernelGGL(k_radix_hist, dim3((unsigned)ntiles), dim3(256), 0, s, kin, n_edges_dev, 8 * p,
                           hist.as<int32_t>(), ntiles);
        run_scan<HistScanOp, int32_t>(HistScanOp{hist.as<int32_t>(), offs.as<int32_t>(), 256 * ntiles},
                                      256 * ntiles, scan, "csc_scan", s);
        hipLaunchKernelGGL(k_radix_scatter, dim3((unsigned)ntiles), dim3(256), 0, s, kin, vin, n_edges_dev, 8 * p,
                           offs.as<int32_t>(), ntiles, kout, vout);
        kin = kout;
        vin = vout;
        cur ^= 1;
    }
    sorted_rows = vin;
    hipLaunchKernelGGL(k_col_ptr, dim3(grid_for(n_src_bound + 1, 256, 4096)), dim3(256), 0, s, kin, n_edges_dev,
                       n_src_bound, col_ptr.as<int32_t>());
    GNNAV_HIP(hipGetLastError());
}

// ----------------------------------------------------- aggregation adjoint
// G lanes per source row; each lane owns Q float4 units of the row.
template <int G, int Q>
__global__ void __launch_bounds__(256) k_aggregate_t(const int32_t *__restrict__ col_ptr,
                                                     const int32_t *__restrict__ col_rows,
                                                     const int32_t *__restrict__ indptr, int64_t n_src,
                                                     const int32_t *__restrict__ n_src_dev, int64_t n_self,
                                                     const int32_t *__restrict__ n_self_dev,
                                                     const f32x4 *__restrict__ dagg, int64_t dagg_ld4,
                                                     const f32x4 *__restrict__ dself, int64_t dself_ld4,
                                                     const f32x4 *__restrict__ mask, int64_t mask_ld4,
                                                     f32x4 *__restrict__ out, int64_t out_ld4, int32_t chunks,
                                                     int32_t d) {
    constexpr int RPW = kWave / G;
    const int lane = lane_id();
    const int sub = lane / G, c0 = lane % G;
    if (n_src_dev) n_src = *n_src_dev;
    if (n_self_dev) n_self = *n_self_dev;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t j = (((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave) * RPW + sub; j < n_src;
         j += nwaves * RPW) {
        const int32_t b = col_ptr[j], e = col_ptr[j + 1];
        for (int32_t slab = 0; slab < chunks; slab += G * Q) {
            f32x4 acc[Q];
            bool live[Q];
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
                live[q] = slab + c0 + q * G < chunks;
            }
            for (int32_t p0 = b; p0 < e; p0 += G) {
                int32_t mine = 0;
                float wmine = 0.0f;
                if (p0 + c0 < e) {
                    mine = col_rows[p0 + c0];
                    wmine = 1.0f / (float)(indptr[mine + 1] - indptr[mine]);
                }
                const int nb = min(G, e - p0);
                for (int k = 0; k < nb; ++k) {
                    const int32_t i = __shfl(mine, k, G);
                    const float w = __shfl(wmine, k, G);
                    const f32x4 *src = dagg + (int64_t)i * dagg_ld4 + slab + c0;
#pragma unroll
                    for (int q = 0; q < Q; ++q)
                        if (live[q]) acc[q] += src[q * G] * w;
                }
            }
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                if (!live[q]) continue;
                const int32_t c = slab + c0 + q * G;
                f32x4 v = acc[q];
                if (dself && j < n_self) v += dself[j * dself_ld4 + c];
                if (mask) {
                    const f32x4 h = mask[j * mask_ld4 + c];
#pragma unroll
                    for (int t = 0; t < 4; ++t) v[t] = h[t] > 0.0f ? v[t] : 0.0f;
                }
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    if (c * 4 + t >= d) v[t] = 0.0f;
                out[j * out_ld4 + c] = v;
            }
        }
    }
}

void launch_aggregate_t(const CscWorkspace &csc, const int32_t *indptr, int64_t n_src, const int32_t *n_src_dev,
                        int64_t n_self, const int32_t *n_self_dev, const float *dagg, int64_t ld_dagg,
                        const float *dself, int64_t ld_dself, const float *mask, int64_t ld_mask, int64_t d,
                        float *out, int64_t ld_out, hipStream_t s, const char *label) {
    if (n_src <= 0) return;
    const int32_t chunks = (int32_t)((d + 3) / 4);
    int g = 1;
    while (g < chunks && g < kWave) g <<= 1;
    int q = (chunks + g - 1) / g;
    if (q > 4) q = 4;
    const unsigned grid = grid_for(n_src, (256 / kWave) * (kWave / g), 8192);
    KernelTimer t(label, s);
#define GNNAV_L(GV, QV)                                                                                          \
    hipLaunchKernelGGL((k_aggregate_t<GV, QV>), dim3(grid), dim3(256), 0, s, csc.col_ptr.as<int32_t>(),            \
                       csc.sorted_rows, indptr, n_src, n_src_dev, n_self, n_self_dev, (const f32x4 *)dagg,         \
                       ld_dagg / 4, (const f32x4 *)dself, ld_dself / 4, (const f32x4 *)mask, ld_mask / 4,         \
                       (f32x4 *)out, ld_out / 4, chunks, (int32_t)d)
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

// --------------------------------------------------------- weight gradient
// Partial tile of dW[seg * d_in + a][o] = sum over the rows m of this split
// of X_seg[m][a] * G[m][o] (rows 16-byte aligned), on the bf16 matrix cores
// through the three-way bf16 split of both operands (bf16split.hpp), so the
// sums carry fp32 rounding.  Both operands move row by row (k = row m)
// straight from global memory into LDS by global_load_lds_dwordx4 through a
// two-stage ring of 32-row steps; LDS holds Xs[m][a] and Gs[m][o] as
// stored.  A wavefront owns (32 VA) x (32 VB) outputs as VA x VB MFMA blocks
// whose rows and columns are interleaved: block (i, j) holds
// a = base + VA r + i and o = base + VB c + j for fragment row r, column c,
// so a lane finds all VA of its X values (and all VB of its G values) for
// one row side by side in LDS, one 4-, 8- or 16-byte read each.  Per 16-row
// sub-step each lane gathers its 8 consecutive rows (k), splits them in
// registers and issues six 32x32x16 bf16 MFMAs per block.  Rows past the
// split's end load a valid row; the lanes that loaded G chunks for them
// zero those in LDS before the barrier, so they add nothing.  Columns past
// d_in or d_out only reach outputs that are not stored.
template <int BA, int BO>
__global__ void __launch_bounds__(256) k_wgrad_split(const float *__restrict__ X0, int64_t ldx0,
                                                     const float *__restrict__ X1, int64_t ldx1, int64_t M,
                                                     const int32_t *__restrict__ m_dev, int64_t d_in,
                                                     const float *__restrict__ Gm, int64_t ldg, int64_t d_out,
                                                     int64_t splits, float *__restrict__ part) {
    typedef float f32x16 __attribute__((ext_vector_type(16)));
    constexpr int BK = 32;
    constexpr int VA = BA / 64, VB = BO / 64;
    constexpr int XC = BA / 4, GC = BO / 4;
    constexpr int X_CH = BK * XC, G_CH = BK * GC, ST = X_CH + G_CH;
    constexpr int X_IN = X_CH / 256, G_IN = G_CH / 256;
    static_assert((VA == 1 || VA == 2 || VA == 4) && (VB == 1 || VB == 2 || VB == 4), "tile");
    static_assert(X_CH % 256 == 0 && G_CH % 256 == 0, "whole wave instructions");
    __shared__ f32x4 S[2 * ST];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wa = wid >> 1, wo = wid & 1, h = lane >> 5, lr = lane & 31;
    if (m_dev) M = *m_dev;
    const int64_t na = (d_in + BA - 1) / BA, no = (d_out + BO - 1) / BO;
    const int64_t tile = blockIdx.x, split = blockIdx.y;
    const int seg = (int)(tile / (na * no));
    const int64_t a0 = ((tile / no) % na) * BA, o0 = (tile % no) * BO;
    const float *X = seg ? X1 : X0;
    const int64_t ldx = seg ? ldx1 : ldx0;
    const int64_t per = ((M + splits - 1) / splits + BK - 1) / BK * BK;
    const int64_t m_lo = split * per, m_hi = std::min<int64_t>(M, m_lo + per);
    const int64_t steps = m_hi > m_lo ? (m_hi - m_lo + BK - 1) / BK : 0;

    f32x16 acc[VA][VB];
#pragma unroll
    for (int i = 0; i < VA; ++i)
#pragma unroll
        for (int j = 0; j < VB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    auto issue = [&](int64_t t) {
        f32x4 *buf = S + (int)(t & 1) * ST;
        const int64_t mb = m_lo + t * BK;
#pragma unroll
        for (int q = 0; q < X_IN; ++q) {
            const int pos = (wid * X_IN + q) * 64 + lane;
            const int64_t m = mb + pos / XC < m_hi ? mb + pos / XC : m_lo;
            const int64_t a = a0 + 4 * (pos % XC);
            dma16(X + m * ldx + (a < d_in ? a : 0), &buf[(wid * X_IN + q) * 64]);
        }
#pragma unroll
        for (int q = 0; q < G_IN; ++q) {
            const int pos = (wid * G_IN + q) * 64 + lane;
            const int64_t m = mb + pos / GC < m_hi ? mb + pos / GC : m_lo;
            const int64_t o = o0 + 4 * (pos % GC);
            dma16(Gm + m * ldg + (o < d_out ? o : 0), &buf[X_CH + (wid * G_IN + q) * 64]);
        }
    };
    auto fixup = [&](int64_t t) {
        const int64_t mb = m_lo + t * BK;
        if (mb + BK <= m_hi) return;
        f32x4 *buf = S + (int)(t & 1) * ST;
#pragma unroll
        for (int q = 0; q < G_IN; ++q) {
            const int pos = (wid * G_IN + q) * 64 + lane;
            if (mb + pos / GC >= m_hi) buf[X_CH + pos] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    typedef float fa_t __attribute__((ext_vector_type(VA)));
    typedef float fb_t __attribute__((ext_vector_type(VB)));
    auto compute = [&](int64_t t) {
        const float *xs = (const float *)(S + (int)(t & 1) * ST);
        const float *gs = xs + 4 * X_CH;
#pragma unroll
        for (int u = 0; u < BK / 16; ++u) {
            float xa[VA][8], xb[VB][8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int row = 16 * u + 8 * h + q;
                const fa_t a = *(const fa_t *)&xs[row * BA + wa * (32 * VA) + VA * lr];
                const fb_t b = *(const fb_t *)&gs[row * BO + wo * (32 * VB) + VB * lr];
#pragma unroll
                for (int i = 0; i < VA; ++i) xa[i][q] = a[i];
#pragma unroll
                for (int j = 0; j < VB; ++j) xb[j][q] = b[j];
            }
            bf16x8 a1[VA], a2[VA], a3[VA], b1[VB], b2[VB], b3[VB];
#pragma unroll
            for (int i = 0; i < VA; ++i) split3(xa[i], a1[i], a2[i], a3[i]);
#pragma unroll
            for (int j = 0; j < VB; ++j) split3(xb[j], b1[j], b2[j], b3[j]);
#pragma unroll
            for (int i = 0; i < VA; ++i)
#pragma unroll
                for (int j = 0; j < VB; ++j)
                    acc[i][j] = mfma_split6(a1[i], a2[i], a3[i], b1[j], b2[j], b3[j], acc[i][j]);
        }
    };
    if (steps > 0) {
        issue(0);
        for (int64_t t = 0; t < steps; ++t) {
            wait_vm<0>();
            fixup(t);
            lds_barrier();           // step t visible; everyone is done with step t - 1
            if (t + 1 < steps) issue(t + 1);
            compute(t);
        }
    }
    float *P = part + split * (2 * d_in * d_out);
#pragma unroll
    for (int i = 0; i < VA; ++i)
#pragma unroll
        for (int j = 0; j < VB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int R = 8 * (r / 4) + 4 * h + (r % 4);
                const int64_t a = a0 + wa * (32 * VA) + VA * R + i;
                const int64_t o = o0 + wo * (32 * VB) + VB * lr + j;
                if (a < d_in && o < d_out) P[(seg * d_in + a) * d_out + o] = acc[i][j][r];
            }
}

// dW = sum of the split partials in split order; optionally copied out, and
// W -= lr * dW when lr != 0.  V = 4: four consecutive elements per lane
// (16-byte loads; total, dw and w 16-byte aligned).  The partials' loads go
// out eight at a time ahead of their adds, which keep the split order.
template <int V>
__global__ void __launch_bounds__(256) k_wgrad_reduce(const float *__restrict__ part, int64_t total, int64_t splits,
                                                      float *__restrict__ dw, float *__restrict__ w, float lr) {
    typedef float fv __attribute__((ext_vector_type(V)));
    const int64_t stride = (int64_t)gridDim.x * blockDim.x, nv = total / V;
    const fv *pv = (const fv *)part;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
        fv g = (fv)0.0f;
        int64_t s = 0;
        for (; s + 8 <= splits; s += 8) {
            fv v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = pv[(s + q) * nv + i];
#pragma unroll
            for (int q = 0; q < 8; ++q) g += v[q];
        }
        for (; s < splits; ++s) g += pv[s * nv + i];
        if (dw) ((fv *)dw)[i] = g;
        if (lr != 0.0f) {
            fv x = ((fv *)w)[i];
            x -= lr * g;
            ((fv *)w)[i] = x;
        }
    }
}

void launch_wgrad(const float *x_self, int64_t ld_self, const float *agg, int64_t ld_agg, int64_t m,
                  const int32_t *m_dev, int64_t d_in, const float *dz, int64_t ld_dz, int64_t d_out, DevBuf &part,
                  float *dw, float *w, float lr, hipStream_t s, const char *label) {
    auto a16 = [](const void *p, int64_t ld) { return (((uintptr_t)p & 15u) == 0) && ld % 4 == 0; };
    if (!(a16(x_self, ld_self) && a16(agg, ld_agg) && a16(dz, ld_dz)))
        fail(GNNAV_E_INVALID, "weight gradient operands need 16-byte aligned rows");
    // 128 x 128 tiles (128 x 64 for outputs at most 64 wide); the row range
    // is split so that at most 512 workgroups run, two per compute unit all
    // at once (rounding up left a few for a second round: 233k layer 1 with
    // 20 tiles ran 520)
    const int64_t BA = 128, BO = d_out > 64 ? 128 : 64;
    const int64_t tiles = 2 * ((d_in + BA - 1) / BA) * ((d_out + BO - 1) / BO);
    int64_t splits = 512 / tiles;
    splits = std::min<int64_t>(splits, std::max<int64_t>(1, (m + 255) / 256));
    splits = std::max<int64_t>(1, std::min<int64_t>(splits, 64));
    const int64_t total = 2 * d_in * d_out;
    part.ensure((size_t)(splits * total) * sizeof(float), s);
    {
        KernelTimer t(label, s);
        if (BO == 128)
            hipLaunchKernelGGL((k_wgrad_split<128, 128>), dim3((unsigned)tiles, (unsigned)splits), dim3(256), 0, s,
                               x_self, ld_self, agg, ld_agg, m, m_dev, d_in, dz, ld_dz, d_out, splits,
                               part.as<float>());
        else
            hipLaunchKernelGGL((k_wgrad_split<128, 64>), dim3((unsigned)tiles, (unsigned)splits), dim3(256), 0, s,
                               x_self, ld_self, agg, ld_agg, m, m_dev, d_in, dz, ld_dz, d_out, splits,
                               part.as<float>());
    }
    {
        KernelTimer t("wgrad_reduce", s);
        const bool vec = total % 4 == 0 && ((uintptr_t)dw & 15u) == 0 && ((uintptr_t)w & 15u) == 0;
        if (vec)
            hipLaunchKernelGGL(k_wgrad_reduce<4>, dim3(grid_for(total / 4, 256, 1024)), dim3(256), 0, s,
                               part.as<float>(), total, splits, dw, w, lr);
        else
            hipLaunchKernelGGL(k_wgrad_reduce<1>, dim3(grid_for(total, 256, 1024)), dim3(256), 0, s,
                               part.as<float>(), total, splits, dw, w, lr);
    }
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
