// Eq. 2 node-wise fanout sampling and the per-hop frontier union.
//
// Per hop h, for 0 < k <= 64 (slot lists):
//   sample       one or more rows per wavefront: copy the row when
//                deg <= k, else Floyd's k-subset with Philox4x32-10 draws;
//                row i writes slots [i s, (i + 1) s) of a slot list,
//                s = min(k, max degree), unused slots -1
//   dedup        first position of each id in the slot list (atomicMin on a
//                dense per-node table, taken by the sample kernel as it
//                writes), then one order-preserving scan of (used, first)
//                pairs compacts the slot list into N_h, writes indptr_h and
//                E_h, appends the new ids to the node list and records their
//                local ids; hop h-1's relabel rides along on extra workgroups
//   relabel      indices_h[p] = local id of N_h[p]
// For other fanouts (k < 0: every neighbour; k > 64) a count scan comes
// first, indptr_h = exclusive scan of min(deg(v), k) over F_(h-1) (for h = 1
// folded into the seeds' dedup scan; for h > 1 carrying hop h-1's relabel),
// the sample kernel writes N_h at those offsets and the dedup scan only
// appends the new ids.
// The node table lives in HBM, one 64-bit entry per graph node:
// (tag << 32) | word with tag = 0xffffffff - (the sampling call's epoch), so
// every entry left by an earlier call compares above every entry of the
// current one and counts as unseen; nothing is cleared between calls.
// Current-call words: the local id (< 2^31) once the node is in the
// frontier, 2^31 + p for the smallest position p seen in the current list.
#include <type_traits>

#include "common.hpp"
#include "scan.hpp"

namespace gnnav {

// ---------------------------------------------------------------- Philox
// Philox4x32-10 (Salmon et al., SC'11): ten rounds; each multiplies words 0
// and 2 by the Philox multipliers and mixes the high halves with words 1, 3
// and the round key; the key advances by the Weyl constants between rounds.
// Only output word 0 is needed.
__device__ __forceinline__ uint32_t philox_word0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                 uint32_t k0, uint32_t k1) {
    constexpr uint32_t kMulA = 0xD2511F53u, kMulB = 0xCD9E8D57u;
    constexpr uint32_t kWeylA = 0x9E3779B9u, kWeylB = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t lo_a = c0 * kMulA, hi_a = __umulhi(c0, kMulA);
        const uint32_t lo_b = c2 * kMulB, hi_b = __umulhi(c2, kMulB);
        const uint32_t x0 = hi_b ^ c1 ^ k0;
        const uint32_t x2 = hi_a ^ c3 ^ k1;
        c0 = x0;
        c1 = lo_b;
        c2 = x2;
        c3 = lo_a;
        k0 += kWeylA;
        k1 += kWeylB;
    }
    return c0;
}

// All four output words (the biased selector uses words 1-3).
__device__ __forceinline__ void philox4(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0, uint32_t k1,
                                        uint32_t (&w)[4]) {
    constexpr uint32_t kMulA = 0xD2511F53u, kMulB = 0xCD9E8D57u;
    constexpr uint32_t kWeylA = 0x9E3779B9u, kWeylB = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t lo_a = c0 * kMulA, hi_a = __umulhi(c0, kMulA);
        const uint32_t lo_b = c2 * kMulB, hi_b = __umulhi(c2, kMulB);
        const uint32_t x0 = hi_b ^ c1 ^ k0;
        const uint32_t x2 = hi_a ^ c3 ^ k1;
        c0 = x0;
        c1 = lo_b;
        c2 = x2;
        c3 = lo_a;
        k0 += kWeylA;
        k1 += kWeylB;
    }
    w[0] = c0;
    w[1] = c1;
    w[2] = c2;
    w[3] = c3;
}

template <class OffT>
__device__ __forceinline__ int64_t row_degree(const OffT *rp, int32_t v, int64_t &start) {
    start = (int64_t)rp[v];
    return (int64_t)rp[v + 1] - start;
}

// The degree of frontier entry v.  Frontier entries are graph nodes; one
// outside [0, n) is only possible after a scan whose look-back wait gave up
// (reported by the next synchronisation point), which can leave stale list
// positions: it counts as a row without neighbours, so no read leaves the
// CSR.
template <class OffT>
__device__ __forceinline__ int64_t frontier_degree(const OffT *rp, int32_t v, int64_t n_nodes, int64_t &start) {
    if (v < 0 || v >= n_nodes) {
        start = 0;
        return 0;
    }
    return row_degree(rp, v, start);
}

// ------------------------------------------------------------ count scan
template <class OffT>
struct CountOp {
    const OffT *row_ptr;
    const int32_t *nodes;
    const int32_t *n_ptr;
    int32_t k;
    int32_t *indptr;
    int32_t *e_out;
    int64_t n_nodes;
    __device__ int64_t n() const { return *n_ptr; }
    __device__ int32_t value(int64_t i) const {
        int64_t st;
        int64_t deg = frontier_degree(row_ptr, nodes[i], n_nodes, st);
        return (int32_t)((k < 0 || deg <= k) ? deg : k);
    }
    __device__ void emit(int64_t i, int32_t prefix, int32_t) const { indptr[i] = prefix; }
    __device__ void total(int32_t t) const {
        indptr[*n_ptr] = t;
        *e_out = t;
    }
};

// Local id of the listed node `id`.  Every listed id is a node of the
// graph and in the frontier by the time this runs, so its node-table entry
// holds a local id below the frontier size.  Anything else is only possible
// after a scan whose look-back wait gave up (reported by the next
// synchronisation point), which can leave list positions unwritten by this
// call: an id outside [0, n) is not looked up, and an entry that is not a
// local id of this frontier becomes 0, so no later kernel reads outside its
// buffers.
__device__ __forceinline__ int32_t local_id(const uint64_t *map, int32_t id, int64_t n_nodes,
                                            const int32_t *n_frontier) {
    if (id < 0 || id >= n_nodes) return 0;
    const uint32_t w = (uint32_t)map[id];
    return w < (uint32_t)*n_frontier ? (int32_t)w : 0;
}

// Local ids of the previous hop's list (its relabel), carried by the count
// scan's launch: both only need that hop's dedup finished.
struct RelabelSide {
    const int32_t *list;
    const int32_t *len_ptr;
    const uint64_t *map;
    int64_t n_nodes;
    const int32_t *n_frontier;
    int32_t *indices;
    __device__ int64_t n() const { return *len_ptr; }
    __device__ void run(int64_t p) const { indices[p] = local_id(map, list[p], n_nodes, n_frontier); }
};

void launch_count_scan(const SampleHopArgs &a, hipStream_t s) {
    auto run = [&](auto op) {
        using Op = decltype(op);
        if (a.relabel_list)
            run_scan<Op, int32_t, RelabelSide>(
                op, a.rows_bound, *a.scan, "count_scan", s,
                RelabelSide{a.relabel_list, a.relabel_len, a.first_map, a.n_nodes, a.relabel_n, a.relabel_indices},
                a.relabel_bound);
        else
            run_scan<Op, int32_t>(op, a.rows_bound, *a.scan, "count_scan", s);
    };
    if (a.offsets_i64)
        run(CountOp<int64_t>{(const int64_t *)a.row_ptr, a.nodes, a.n_prev, a.fanout, a.indptr, a.e_out, a.n_nodes});
    else
        run(CountOp<int32_t>{(const int32_t *)a.row_ptr, a.nodes, a.n_prev, a.fanout, a.indptr, a.e_out, a.n_nodes});
}

__device__ __forceinline__ uint64_t node_position(uint32_t tag, int64_t p) {
    return ((uint64_t)tag << 32) | (0x80000000ull + (uint64_t)p);
}
__device__ __forceinline__ uint64_t node_local(uint32_t tag, int64_t local) {
    return ((uint64_t)tag << 32) | (uint64_t)local;
}

// First position of `id` in the hop's list: a position only ever lowers a
// stale entry or a larger position of this call (frontier entries are
// smaller than every position), and the read skips most of the atomics.
__device__ __forceinline__ void note_first(unsigned long long *map, uint32_t tag, int32_t id, int64_t pos) {
    const unsigned long long e = node_position(tag, pos);
    if (map && map[id] > e) atomicMin(&map[id], e);
}

// ---------------------------------------------------------- sample kernel
// One wavefront per destination row, grid-stride over rows.  For k <= 64
// lane j holds draw j: t_j = floor(x_j * (m_j + 1) / 2^32), m_j = deg-k+j.
// Floyd's rule is sequential in j (slot j takes t_j unless an earlier slot
// already holds it, then m_j), so the wave walks j in order and decides
// each slot with one ballot against the slots already fixed.
template <class OffT>
__global__ void __launch_bounds__(256) k_sample_small(const OffT *__restrict__ row_ptr,
                                                      const int32_t *__restrict__ col,
                                                      const int32_t *__restrict__ nodes,
                                                      const int32_t *__restrict__ n_prev,
                                                      const int32_t *__restrict__ indptr,
                                                      int32_t *__restrict__ out, int32_t k,
                                                      uint32_t key0, uint32_t key1, uint32_t hop,
                                                      unsigned long long *__restrict__ first, uint32_t tag,
                                                      int32_t stride, int64_t n_nodes) {
    const int lane = lane_id();
    const int64_t n_rows = *n_prev;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; i < n_rows; i += nwaves) {
        const int32_t v = nodes[i];
        int64_t start;
        const int64_t deg = frontier_degree(row_ptr, v, n_nodes, start);
        const int64_t at = stride ? i * stride : (int64_t)indptr[i];
        int32_t *dst = out + at;
        if (k < 0 || deg <= k) {
            for (int64_t j = lane; j < deg; j += kWave) {
                const int32_t id = col[start + j];
                dst[j] = id;
                note_first(first, tag, id, at + j);
            }
            for (int64_t j = deg + lane; j < stride; j += kWave) dst[j] = -1;
            continue;
        }
        uint32_t t = 0, m = 0;
        if (lane < k) {
            m = (uint32_t)(deg - k + lane);
            const uint32_t x = philox_word0((uint32_t)lane, (uint32_t)v, 0u, hop, key0, key1);
            t = __umulhi(x, m + 1u);
        }
        uint32_t pick = t;
        for (int j = 1; j < k; ++j) {
            const uint32_t tj = (uint32_t)__builtin_amdgcn_readlane((int)t, j);
            const uint64_t clash = __ballot(lane < j && pick == tj);
            if (lane == j && clash != 0) pick = m;
        }
        if (lane < k) {
            const int32_t id = col[start + pick];
            dst[lane] = id;
            note_first(first, tag, id, at + lane);
        }
    }
}

// 0 < k <= G <= 32: the same selection with G lanes per row, 64 / G rows
// per wavefront (a hop's fanout is uniform, so the rows of a wavefront walk
// the same j loop; lane j of a row reads t_j of its own row by a width-G
// shuffle and tests the row's bits of one ballot).
template <class OffT, int G>
__global__ void __launch_bounds__(256) k_sample_group(const OffT *__restrict__ row_ptr,
                                                      const int32_t *__restrict__ col,
                                                      const int32_t *__restrict__ nodes,
                                                      const int32_t *__restrict__ n_prev,
                                                      const int32_t *__restrict__ indptr,
                                                      int32_t *__restrict__ out, int32_t k,
                                                      uint32_t key0, uint32_t key1, uint32_t hop,
                                                      unsigned long long *__restrict__ first, uint32_t tag,
                                                      int32_t stride, int64_t n_nodes) {
    constexpr int R = kWave / G;
    const int lane = lane_id(), r = lane / G, gl = lane % G;
    const int64_t n_rows = *n_prev;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t base = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave * R; base < n_rows;
         base += nwaves * R) {
        const int64_t i = base + r;
        const bool valid = i < n_rows;
        int32_t v = 0;
        int64_t start = 0, deg = 0, at = 0;
        if (valid) {
            v = nodes[i];
            deg = frontier_degree(row_ptr, v, n_nodes, start);
            at = stride ? i * stride : (int64_t)indptr[i];
        }
        const bool draw = valid && deg > k;
        uint32_t t = 0, m = 0;
        if (draw && gl < k) {
            m = (uint32_t)(deg - k + gl);
            const uint32_t x = philox_word0((uint32_t)gl, (uint32_t)v, 0u, hop, key0, key1);
            t = __umulhi(x, m + 1u);
        }
        uint32_t pick = t;
        for (int j = 1; j < k; ++j) {
            const uint32_t tj = (uint32_t)__shfl((int)t, j, G);
            const uint64_t clash = (__ballot(gl < j && pick == tj) >> (r * G)) & ((1ull << j) - 1ull);
            if (gl == j && clash != 0) pick = m;
        }
        const bool writes = draw ? gl < k : (valid && gl < deg);
        if (writes) {
            const int32_t id = col[start + (draw ? (int64_t)pick : (int64_t)gl)];
            out[at + gl] = id;
            note_first(first, tag, id, at + gl);
        } else if (valid && gl < stride) {
            out[at + gl] = -1;
        }
    }
}

// 64 < k <= kMaxFanout: chosen offsets kept in LDS per wave; each slot j is
// checked against all earlier slots with a wave-wide ballot per 64 slots.
constexpr int kMaxFanout = 1024;

template <class OffT>
__global__ void __launch_bounds__(256) k_sample_big(const OffT *__restrict__ row_ptr,
                                                    const int32_t *__restrict__ col,
                                                    const int32_t *__restrict__ nodes,
                                                    const int32_t *__restrict__ n_prev,
                                                    const int32_t *__restrict__ indptr,
                                                    int32_t *__restrict__ out, int32_t k,
                                                    uint32_t key0, uint32_t key1, uint32_t hop,
                                                    unsigned long long *__restrict__ first, uint32_t tag,
                                                    int32_t stride, int64_t n_nodes) {
    __shared__ uint32_t taken_all[256 / kWave][kMaxFanout];
    uint32_t *taken = taken_all[threadIdx.x / kWave];
    const int lane = lane_id();
    const int64_t n_rows = *n_prev;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; i < n_rows; i += nwaves) {
        const int32_t v = nodes[i];
        int64_t start;
        const int64_t deg = frontier_degree(row_ptr, v, n_nodes, start);
        const int64_t at = stride ? i * stride : (int64_t)indptr[i];
        int32_t *dst = out + at;
        if (deg <= k) {
            for (int64_t j = lane; j < deg; j += kWave) {
                const int32_t id = col[start + j];
                dst[j] = id;
                note_first(first, tag, id, at + j);
            }
            for (int64_t j = deg + lane; j < stride; j += kWave) dst[j] = -1;
            continue;
        }
        for (int jb = 0; jb < k; jb += kWave) {
            const int jl = jb + lane;
            uint32_t t = 0, m = 0;
            if (jl < k) {
                m = (uint32_t)(deg - k + jl);
                const uint32_t x = philox_word0((uint32_t)jl, (uint32_t)v, 0u, hop, key0, key1);
                t = __umulhi(x, m + 1u);
            }
            uint32_t pick = t;
            const int jend = min(k, jb + kWave);
            for (int j = jb; j < jend; ++j) {
                const uint32_t tj = (uint32_t)__builtin_amdgcn_readlane((int)t, j - jb);
                bool hit = lane < j - jb && pick == tj;
                for (int q = lane; q < jb; q += kWave) hit = hit || taken[q] == tj;
                const uint64_t clash = __ballot(hit);
                if (lane == j - jb && clash != 0) pick = m;
            }
            if (jl < k) taken[jl] = pick;
            __builtin_amdgcn_s_waitcnt(0);
            __builtin_amdgcn_wave_barrier();
        }
        for (int q = lane; q < k; q += kWave) {
            const int32_t id = col[start + taken[q]];
            dst[q] = id;
            note_first(first, tag, id, at + q);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// Locality-biased selection (k <= 64), one wavefront per row.  Cached
// neighbours (slot_map >= 0) weigh eta, the others 1; the k picks follow
// successive sampling without replacement, done as
//   1. the class of pick j = 0..k-1, in order: with c_r cached and u_r
//      uncached left, t = floor(x * (eta*c_r + u_r) / 2^32), x = Philox word
//      1 of counter (j, v, hop); cached when t < eta*c_r;
//   2. Floyd's uniform subset inside each class: lane j < kc runs cached step
//      j with word 2 of counter (j, v, hop), lane kc + j runs uncached step j
//      with word 3 of counter (j, v, hop);
//   3. the chosen class indices are mapped to row offsets by walking the row
//      in 64-neighbour chunks with a ballot of the cached flags.
// Output: cached picks in Floyd order, then the uncached ones.
template <class OffT>
__global__ void __launch_bounds__(256) k_sample_biased(const OffT *__restrict__ row_ptr,
                                                       const int32_t *__restrict__ col,
                                                       const int32_t *__restrict__ nodes,
                                                       const int32_t *__restrict__ n_prev,
                                                       const int32_t *__restrict__ indptr,
                                                       int32_t *__restrict__ out, int32_t k, uint32_t key0,
                                                       uint32_t key1, uint32_t hop,
                                                       const int32_t *__restrict__ slot_map, uint32_t eta,
                                                       const int32_t *__restrict__ part_col,
                                                       const int32_t *__restrict__ part_cnt,
                                                       unsigned long long *__restrict__ first, uint32_t tag,
                                                       int32_t stride, int64_t n_nodes) {
    const int lane = lane_id();
    const int64_t n_rows = *n_prev;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; i < n_rows; i += nwaves) {
        const int32_t v = nodes[i];
        int64_t start;
        const int64_t deg = frontier_degree(row_ptr, v, n_nodes, start);
        const int64_t at = stride ? i * stride : (int64_t)indptr[i];
        int32_t *dst = out + at;
        if (k < 0 || deg <= k) {
            for (int64_t j = lane; j < deg; j += kWave) {
                const int32_t id = col[start + j];
                dst[j] = id;
                note_first(first, tag, id, at + j);
            }
            for (int64_t j = deg + lane; j < stride; j += kWave) dst[j] = -1;
            continue;
        }
        // cached neighbours of the row
        int64_t c = 0;
        if (part_cnt) {
            c = part_cnt[v];
        } else {
            for (int64_t base = 0; base < deg; base += kWave) {
                const bool f = base + lane < deg && slot_map[col[start + base + lane]] >= 0;
                c += __popcll(__ballot(f));
            }
        }
        const int64_t u = deg - c;
        // 1. classes
        uint32_t w[4];
        philox4((uint32_t)lane, (uint32_t)v, 0u, hop, key0, key1, w);
        const uint32_t x1 = w[1];
        int64_t cr = c, ur = u;
        int32_t kc = 0;
        for (int j = 0; j < k; ++j) {
            const uint32_t x = (uint32_t)__builtin_amdgcn_readlane((int)x1, j);
            const uint64_t heavy = (uint64_t)eta * (uint64_t)cr;
            const uint64_t b = heavy + (uint64_t)ur;
            const uint64_t t = (uint64_t)x * (b >> 32) + (((uint64_t)x * (b & 0xffffffffull)) >> 32);
            if (t < heavy) {
                ++kc;
                --cr;
            } else {
                --ur;
            }
        }
        // 2. Floyd inside each class
        const bool cached_lane = lane < kc;
        const int32_t step = cached_lane ? lane : lane - kc;
        const int64_t size = cached_lane ? c : u, kk = cached_lane ? kc : k - kc;
        uint32_t t = 0, m = 0;
        if (lane < k) {
            philox4((uint32_t)step, (uint32_t)v, 0u, hop, key0, key1, w);
            m = (uint32_t)(size - kk + step);
            t = __umulhi(cached_lane ? w[2] : w[3], m + 1u);
        }
        uint32_t pick = t;
        for (int j = 1; j < k; ++j) {
            const uint32_t tj = (uint32_t)__builtin_amdgcn_readlane((int)t, j);
            const bool same = (lane < kc) == (j < kc);
            const uint64_t clash = __ballot(same && lane < j && pick == tj);
            if (lane == j && clash != 0) pick = m;
        }
        // 3. class index -> row offset
        if (part_col) {
            if (lane < k) {
                const int32_t id = part_col[start + (cached_lane ? 0 : c) + pick];
                dst[lane] = id;
                note_first(first, tag, id, at + lane);
            }
            continue;
        }
        int64_t seen = 0, pos = -1;
        bool need = lane < k;
        for (int64_t base = 0; base < deg && __ballot(need) != 0; base += kWave) {
            const bool valid = base + lane < deg;
            const bool f = valid && slot_map[col[start + base + lane]] >= 0;
            const uint64_t mc = __ballot(f), mu = __ballot(valid && !f);
            uint64_t mask = cached_lane ? mc : mu;
            const int64_t cnt = __popcll(mask);
            if (need && (int64_t)pick < seen + cnt) {
                for (int64_t r = (int64_t)pick - seen; r > 0; --r) mask &= mask - 1;
                pos = base + __builtin_ctzll(mask);
                need = false;
            }
            seen += cnt;
        }
        if (lane < k) {
            const int32_t id = col[start + (pos < 0 ? 0 : pos)];   // pos >= 0 whenever pick < class size
            dst[lane] = id;
            note_first(first, tag, id, at + lane);
        }
    }
}

// Each row's neighbours split into cached then uncached, CSR order kept
// within each class; part_cnt[v] = cached neighbours of v.  One wavefront
// per row: a ballot per 64 neighbours gives every lane its rank in its class.
template <class OffT>
__global__ void __launch_bounds__(256) k_partition_rows(const OffT *__restrict__ row_ptr,
                                                        const int32_t *__restrict__ col, int64_t n,
                                                        const int32_t *__restrict__ slot_map,
                                                        int32_t *__restrict__ part_col, int32_t *__restrict__ part_cnt) {
    const int lane = lane_id();
    const uint64_t below = (1ull << lane) - 1ull;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t v = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; v < n; v += nwaves) {
        int64_t start;
        const int64_t deg = row_degree(row_ptr, (int32_t)v, start);
        int64_t c = 0;
        for (int64_t base = 0; base < deg; base += kWave) {
            const bool f = base + lane < deg && slot_map[col[start + base + lane]] >= 0;
            c += __popcll(__ballot(f));
        }
        int64_t seen_c = 0, seen_u = 0;
        for (int64_t base = 0; base < deg; base += kWave) {
            const bool valid = base + lane < deg;
            const int32_t x = valid ? col[start + base + lane] : 0;
            const bool f = valid && slot_map[x] >= 0;
            const uint64_t mc = __ballot(f), mu = __ballot(valid && !f);
            if (valid) {
                const int64_t at = f ? seen_c + __popcll(mc & below) : c + seen_u + __popcll(mu & below);
                part_col[start + at] = x;
            }
            seen_c += __popcll(mc);
            seen_u += __popcll(mu);
        }
        if (lane == 0) part_cnt[v] = (int32_t)c;
    }
}

void launch_partition_rows(const void *row_ptr, bool offsets_i64, const int32_t *col, int64_t n,
                           const int32_t *slot_map, int32_t *part_col, int32_t *part_cnt, hipStream_t s) {
    if (n <= 0) return;
    const unsigned grid = grid_for(n, 256 / kWave, 16384);
    KernelTimer t("partition_rows", s);
    if (offsets_i64)
        hipLaunchKernelGGL(k_partition_rows<int64_t>, dim3(grid), dim3(256), 0, s, (const int64_t *)row_ptr, col, n,
                           slot_map, part_col, part_cnt);
    else
        hipLaunchKernelGGL(k_partition_rows<int32_t>, dim3(grid), dim3(256), 0, s, (const int32_t *)row_ptr, col, n,
                           slot_map, part_col, part_cnt);
    GNNAV_HIP(hipGetLastError());
}

void launch_sample_hop(const SampleHopArgs &a, hipStream_t s) {
    if (a.rows_bound <= 0) return;
    if (a.bias_slot_map) {
        GNNAV_CHECK(a.fanout <= kWave, GNNAV_E_INVALID, "biased sampling supports fanouts up to 64");
        GNNAV_CHECK(a.slot_stride == 0 || (a.fanout > 0 && a.slot_stride <= a.fanout), GNNAV_E_INVALID,
                    "slot lists need 0 < slot stride <= fanout");
        const uint32_t key0 = (uint32_t)(a.rng_seed & 0xffffffffu), key1 = (uint32_t)(a.rng_seed >> 32);
        const unsigned grid = grid_for(a.rows_bound, 256 / kWave, 16384);
        KernelTimer t("sample_hop", s);
        if (a.offsets_i64)
            hipLaunchKernelGGL(k_sample_biased<int64_t>, dim3(grid), dim3(256), 0, s, (const int64_t *)a.row_ptr, a.col,
                               a.nodes, a.n_prev, a.indptr, a.nbrs, a.fanout, key0, key1, a.hop, a.bias_slot_map,
                               a.eta, a.part_col, a.part_cnt, (unsigned long long *)a.first_map, a.map_tag,
                               a.slot_stride, a.n_nodes);
        else
            hipLaunchKernelGGL(k_sample_biased<int32_t>, dim3(grid), dim3(256), 0, s, (const int32_t *)a.row_ptr, a.col,
                               a.nodes, a.n_prev, a.indptr, a.nbrs, a.fanout, key0, key1, a.hop, a.bias_slot_map,
                               a.eta, a.part_col, a.part_cnt, (unsigned long long *)a.first_map, a.map_tag,
                               a.slot_stride, a.n_nodes);
        GNNAV_HIP(hipGetLastError());
        return;
    }
    GNNAV_CHECK(a.fanout <= kMaxFanout, GNNAV_E_INVALID, "fanout above 1024");
    GNNAV_CHECK(a.slot_stride == 0 || (a.fanout > 0 && a.fanout <= kWave && a.slot_stride <= a.fanout),
                GNNAV_E_INVALID, "slot lists need 0 < slot stride <= fanout <= 64");
    const uint32_t key0 = (uint32_t)(a.rng_seed & 0xffffffffu), key1 = (uint32_t)(a.rng_seed >> 32);
    const unsigned grid = grid_for(a.rows_bound, 256 / kWave, 16384);
    KernelTimer t("sample_hop", s);
    auto first = (unsigned long long *)a.first_map;
    auto run = [&](auto row_ptr) {
        using OffT = std::remove_const_t<std::remove_pointer_t<decltype(row_ptr)>>;
        const int k = a.fanout;
        auto group = [&](auto kern, int rows_per_wave) {
            hipLaunchKernelGGL(kern, dim3(grid_for(a.rows_bound, (256 / kWave) * rows_per_wave, 16384)), dim3(256), 0,
                               s, row_ptr, a.col, a.nodes, a.n_prev, a.indptr, a.nbrs, k, key0, key1, a.hop, first,
                               a.map_tag, a.slot_stride, a.n_nodes);
        };
        if (k > 0 && k <= 8)
            group(k_sample_group<OffT, 8>, 8);
        else if (k > 0 && k <= 16)
            group(k_sample_group<OffT, 16>, 4);
        else if (k > 0 && k <= 32)
            group(k_sample_group<OffT, 32>, 2);
        else
            hipLaunchKernelGGL(k > kWave ? k_sample_big<OffT> : k_sample_small<OffT>, dim3(grid), dim3(256), 0, s,
                               row_ptr, a.col, a.nodes, a.n_prev, a.indptr, a.nbrs, k, key0, key1, a.hop, first,
                               a.map_tag, a.slot_stride, a.n_nodes);
    };
    if (a.offsets_i64)
        run((const int64_t *)a.row_ptr);
    else
        run((const int32_t *)a.row_ptr);
    GNNAV_HIP(hipGetLastError());
}

// ------------------------------------------------------------------ dedup
__device__ __forceinline__ int64_t list_len(int64_t c, const int32_t *p) { return p ? (int64_t)*p : c; }

// First positions of a list's ids in the node table; out-of-range ids are
// counted into *err.  err_next (nullable) is the count slot of the next call
// on the same blocks, cleared here so that no separate launch has to clear a
// slot before each call (its previous value was reported by the call that
// used it).
__global__ void __launch_bounds__(256) k_first_position(const int32_t *__restrict__ list, int64_t len_const,
                                                        const int32_t *__restrict__ len_ptr,
                                                        unsigned long long *__restrict__ map, uint32_t tag,
                                                        int64_t n_nodes, int32_t *__restrict__ err,
                                                        int32_t *__restrict__ err_next) {
    const int64_t len = list_len(len_const, len_ptr);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    if (err_next && blockIdx.x == 0 && threadIdx.x == 0) *err_next = 0;
    int32_t bad = 0;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < len; p += stride) {
        const int32_t id = list[p];
        if (id < 0 || id >= n_nodes) {
            ++bad;
            continue;
        }
        note_first(map, tag, id, p);
    }
    if (bad && err) atomicAdd(err, bad);
}

// The seeds' dedup when they fit one scan tile (at most kScanTile ids, no
// frontier before them, no folded count scan): first positions and the
// order-preserving scan of first-occurrence flags in one workgroup, which
// saves the separate first-position launch.  Between the two phases every
// wavefront waits for its node-table atomics to be performed in L2, then
// the workgroup meets at a barrier; the flags then read the table with
// device-scope loads, past the compute unit's cache, which may hold lines
// read before the atomics.  Results equal those of k_first_position
// followed by the DedupOp scan.
__global__ void __launch_bounds__(kScanThreads) k_seed_dedup_tile(const int32_t *__restrict__ list, int64_t len,
                                                                  unsigned long long *__restrict__ map, uint32_t tag,
                                                                  int64_t n_nodes, int32_t *__restrict__ nodes,
                                                                  int32_t *__restrict__ size_out,
                                                                  int32_t *__restrict__ err,
                                                                  int32_t *__restrict__ err_next) {
    __shared__ int32_t scratch[kScanThreads / kWave];
    __shared__ int32_t s_bad;
    if (threadIdx.x == 0) {
        s_bad = 0;
        if (err_next) *err_next = 0;
    }
    __syncthreads();
    const int64_t first = (int64_t)threadIdx.x * kScanItems;
    // every load of a phase issued before any of its results is used
    int32_t ids[kScanItems];
    bool ok[kScanItems];
    int32_t bad = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) ids[j] = first + j < len ? list[first + j] : -1;
    unsigned long long cur[kScanItems];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        ok[j] = first + j < len && ids[j] >= 0 && ids[j] < n_nodes;
        bad += first + j < len && !ok[j];
        cur[j] = ok[j] ? map[ids[j]] : 0ull;
    }
    // a position only lowers a stale entry or a larger position of this call
    bool lower[kScanItems];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) lower[j] = ok[j] && cur[j] > node_position(tag, first + j);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j)
        if (lower[j]) atomicMin(&map[ids[j]], node_position(tag, first + j));
    if (bad) atomicAdd(&s_bad, bad);
    __builtin_amdgcn_s_waitcnt(0);   // vmcnt(0), lgkmcnt(0): this wavefront's atomics are done
    __syncthreads();
    if (threadIdx.x == 0 && s_bad && err) atomicAdd(err, s_bad);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j)
        cur[j] = ok[j] ? __hip_atomic_load(&map[ids[j]], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0ull;
    int32_t flag[kScanItems], cnt = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        flag[j] = ok[j] && cur[j] == node_position(tag, first + j);
        cnt += flag[j];
    }
    int32_t total;
    int32_t at = block_exclusive_sum<int32_t, kScanThreads>(cnt, scratch, total);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        if (!flag[j]) continue;
        nodes[at] = ids[j];
        map[ids[j]] = node_local(tag, at);
        ++at;
    }
    if (threadIdx.x == 0) *size_out = total;
}

struct DedupOp {
    const int32_t *list;
    int64_t len_const;
    const int32_t *len_ptr;
    unsigned long long *map;
    uint32_t tag;
    int64_t n_nodes;
    int32_t *nodes;
    const int32_t *base_ptr;
    int32_t *size_out;
    // the id and whether p is its first position, read once for both passes
    struct Item {
        int32_t id, first;
    };
    __device__ int64_t n() const { return list_len(len_const, len_ptr); }
    __device__ Item load(int64_t p) const {
        const int32_t id = list[p];
        if (id < 0 || id >= n_nodes) return Item{id, 0};
        return Item{id, map[id] == node_position(tag, p) ? 1 : 0};
    }
    __device__ int32_t value(const Item &it) const { return it.first; }
    __device__ void emit(int64_t p, int32_t prefix, int32_t v, const Item &it) const {
        if (!v) return;
        const int32_t local = (base_ptr ? *base_ptr : 0) + prefix;
        nodes[local] = it.id;
        map[it.id] = node_local(tag, local);
    }
    __device__ void total(int32_t t) const { *size_out = (base_ptr ? *base_ptr : 0) + t; }
};

// The seeds' dedup with hop 1's count scan folded in: F_0 is exactly the
// seeds' first occurrences in order, so one scan of (first, min(deg, k))
// pairs gives both the local ids and indptr_1 (edges in the high half).
template <class OffT>
struct SeedDedupCountOp {
    DedupOp d;
    const OffT *row_ptr;
    int32_t k;
    int32_t *indptr;
    int32_t *e_out;
    struct Item {
        int32_t id, first, count;
    };
    __device__ int64_t n() const { return d.n(); }
    __device__ Item load(int64_t p) const {
        const DedupOp::Item b = d.load(p);
        int32_t c = 0;
        if (b.first) {
            int64_t st;
            const int64_t deg = row_degree(row_ptr, b.id, st);
            c = (int32_t)((k < 0 || deg <= k) ? deg : k);
        }
        return Item{b.id, b.first, c};
    }
    __device__ int64_t value(const Item &it) const { return ((int64_t)it.count << 32) | (int64_t)it.first; }
    __device__ void emit(int64_t p, int64_t prefix, int64_t v, const Item &it) const {
        if (!it.first) return;
        const int32_t local = (int32_t)(prefix & 0xffffffff);
        d.nodes[local] = it.id;
        d.map[it.id] = node_local(d.tag, local);
        indptr[local] = (int32_t)(prefix >> 32);
    }
    __device__ void total(int64_t t) const {
        const int32_t nf = (int32_t)(t & 0xffffffff), e = (int32_t)(t >> 32);
        *d.size_out = nf;
        indptr[nf] = e;
        *e_out = e;
    }
};

// The dedup of a slot list (rows of `stride` slots, -1 where unused), with
// the list's compaction folded in: one scan of (used, first) pairs, the used
// count in the high half, gives every used slot its position in N_h, every
// row its offset (the prefix at its first slot) and every first occurrence
// its local id.  The slot list is in row order, so N_h keeps the order of
// the rows and, within a row, of the picks.
struct DedupCompactOp {
    const int32_t *slots;
    const int32_t *rows_ptr;   // device: rows (= |F_(h-1)|, also the local id base)
    int32_t stride;
    unsigned long long *map;
    uint32_t tag;
    int64_t n_nodes;
    int32_t *nodes;
    int32_t *size_out;
    int32_t *compact;
    int32_t *indptr;
    int32_t *e_out;
    struct Item {
        int32_t id, used, first;
    };
    __device__ int64_t n() const { return (int64_t)*rows_ptr * stride; }
    __device__ Item load(int64_t p) const {
        const int32_t id = slots[p];
        if (id < 0 || id >= n_nodes) return Item{id, 0, 0};
        return Item{id, 1, map[id] == node_position(tag, p) ? 1 : 0};
    }
    __device__ int64_t value(const Item &it) const { return ((int64_t)it.used << 32) | (int64_t)it.first; }
    __device__ void emit(int64_t p, int64_t prefix, int64_t, const Item &it) const {
        const int32_t at = (int32_t)(prefix >> 32);
        const int64_t row = p / stride;
        if (row * stride == p) indptr[row] = at;
        if (!it.used) return;
        compact[at] = it.id;
        if (it.first) {
            const int32_t local = *rows_ptr + (int32_t)(prefix & 0xffffffff);
            nodes[local] = it.id;
            map[it.id] = node_local(tag, local);
        }
    }
    __device__ void total(int64_t t) const {
        const int32_t e = (int32_t)(t >> 32), rows = *rows_ptr;
        indptr[rows] = e;
        *e_out = e;
        *size_out = rows + (int32_t)(t & 0xffffffff);
    }
};

void launch_dedup(const DedupArgs &a, hipStream_t s) {
    if (!a.first_done && !a.len_ptr && !a.base_ptr && !a.count_row_ptr && a.slot_stride == 0 &&
        a.len_const <= kScanTile) {
        KernelTimer t("dedup_scan", s);
        hipLaunchKernelGGL(k_seed_dedup_tile, dim3(1), dim3(kScanThreads), 0, s, a.list, a.len_const,
                           (unsigned long long *)a.map, a.tag, a.n_nodes, a.nodes, a.size_out, a.err, a.err_next);
        GNNAV_HIP(hipGetLastError());
        return;
    }
    if ((a.len_bound > 0 || a.err_next) && !a.first_done) {
        KernelTimer t("dedup_first", s);
        hipLaunchKernelGGL(k_first_position, dim3(grid_for(a.len_bound, 256, 8192)), dim3(256), 0, s,
                           a.list, a.len_const, a.len_ptr, (unsigned long long *)a.map, a.tag, a.n_nodes, a.err,
                           a.err_next);
        GNNAV_HIP(hipGetLastError());
    }
    if (a.slot_stride > 0) {
        GNNAV_CHECK(a.first_done && a.base_ptr && a.compact_out && a.indptr_out && a.e_out, GNNAV_E_INVALID,
                    "a slot list's dedup needs its sampler's first positions, row count and outputs");
        DedupCompactOp op{a.list, a.base_ptr, a.slot_stride, (unsigned long long *)a.map, a.tag, a.n_nodes,
                          a.nodes, a.size_out, a.compact_out, a.indptr_out, a.e_out};
        if (a.relabel_list)
            run_scan<DedupCompactOp, int64_t, RelabelSide>(
                op, a.len_bound, *a.scan, "dedup_scan", s,
                RelabelSide{a.relabel_list, a.relabel_len, a.map, a.n_nodes, a.relabel_n, a.relabel_indices},
                a.relabel_bound);
        else
            run_scan<DedupCompactOp, int64_t>(op, a.len_bound, *a.scan, "dedup_scan", s);
        return;
    }
    DedupOp op{a.list, a.len_const, a.len_ptr, (unsigned long long *)a.map, a.tag, a.n_nodes, a.nodes, a.base_ptr,
               a.size_out};
    if (a.count_row_ptr) {
        GNNAV_CHECK(!a.base_ptr, GNNAV_E_INVALID, "a folded count scan needs an empty frontier before the list");
        if (a.count_i64)
            run_scan<SeedDedupCountOp<int64_t>, int64_t>(
                SeedDedupCountOp<int64_t>{op, (const int64_t *)a.count_row_ptr, a.count_k, a.count_indptr, a.count_e_out},
                a.len_bound, *a.scan, "dedup_scan", s);
        else
            run_scan<SeedDedupCountOp<int32_t>, int64_t>(
                SeedDedupCountOp<int32_t>{op, (const int32_t *)a.count_row_ptr, a.count_k, a.count_indptr, a.count_e_out},
                a.len_bound, *a.scan, "dedup_scan", s);
        return;
    }
    run_scan<DedupOp, int32_t>(op, a.len_bound, *a.scan, "dedup_scan", s);
}

__global__ void __launch_bounds__(256) k_relabel(const int32_t *__restrict__ list,
                                                 const int32_t *__restrict__ len_ptr,
                                                 const uint64_t *__restrict__ map, int64_t n_nodes,
                                                 const int32_t *__restrict__ n_frontier,
                                                 int32_t *__restrict__ indices) {
    const int64_t len = *len_ptr;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < len; p += stride)
        indices[p] = local_id(map, list[p], n_nodes, n_frontier);
}

void launch_relabel(const int32_t *list, const int32_t *len_ptr, int64_t len_bound, const uint64_t *map,
                    int64_t n_nodes, const int32_t *n_frontier, int32_t *indices, hipStream_t s) {
    if (len_bound <= 0) return;
    KernelTimer t("relabel", s);
    hipLaunchKernelGGL(k_relabel, dim3(grid_for(len_bound, 256, 8192)), dim3(256), 0, s, list, len_ptr,
                       map, n_nodes, n_frontier, indices);
    GNNAV_HIP(hipGetLastError());
}

__global__ void __launch_bounds__(256) k_fill_i32(int32_t *__restrict__ p, int32_t v, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

void launch_fill_i32(int32_t *p, int32_t v, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256, 8192)), dim3(256), 0, s, p, v, n);
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
