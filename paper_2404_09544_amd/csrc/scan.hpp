// Device-wide exclusive scan with a per-element emit step.
//
// An Op supplies, on the device:
//   int64_t n() const                    element count (may be read from HBM)
//   V value(int64_t i) const             contribution of element i
//   void emit(int64_t i, V prefix, V v)  called for every i with its
//                                        exclusive prefix (sum over j < i)
//   void total(V t)                      called once with the grand total
// Three launches: per-tile sums, one block scanning the tile sums into tile
// offsets (and reporting the total), then per-tile scans that emit.  Each
// thread owns kItems consecutive elements, so the emit order inside a tile
// follows the element order and the result does not depend on scheduling.
#pragma once

#include "common.hpp"

namespace gnnav {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

template <class Op, class V>
__global__ void __launch_bounds__(kScanThreads) k_scan_tiles(Op op, V *part) {
    __shared__ V scratch[kScanThreads / kWave];
    const int64_t n = op.n();
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    if (base >= n) return;  // uniform across the block
    const int64_t first = base + (int64_t)threadIdx.x * kScanItems;
    V s = V(0);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        int64_t i = first + j;
        if (i < n) s += op.value(i);
    }
    V total;
    block_exclusive_sum<V, kScanThreads>(s, scratch, total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

template <class Op, class V>
__global__ void __launch_bounds__(1024) k_scan_spine(Op op, V *part) {
    __shared__ V scratch[1024 / kWave];
    const int64_t n = op.n();
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    V carry = V(0);
    for (int64_t b = 0; b < tiles; b += 1024) {
        int64_t i = b + threadIdx.x;
        V x = i < tiles ? part[i] : V(0);
        V total;
        V ex = block_exclusive_sum<V, 1024>(x, scratch, total);
        if (i < tiles) part[i] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0) op.total(carry);
}

template <class Op, class V>
__global__ void __launch_bounds__(kScanThreads) k_scan_emit(Op op, const V *part) {
    __shared__ V scratch[kScanThreads / kWave];
    const int64_t n = op.n();
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    if (base >= n) return;
    const int64_t first = base + (int64_t)threadIdx.x * kScanItems;
    V vals[kScanItems];
    V s = V(0);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        int64_t i = first + j;
        vals[j] = i < n ? op.value(i) : V(0);
        s += vals[j];
    }
    V total;
    V run = block_exclusive_sum<V, kScanThreads>(s, scratch, total) + part[blockIdx.x];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        int64_t i = first + j;
        if (i < n) op.emit(i, run, vals[j]);
        run += vals[j];
    }
}

// Enqueue the three launches.  `bound` >= op.n() sizes the grids; `part`
// must hold ceil(bound / kScanTile) values (at least one).
template <class Op, class V>
void run_scan(const Op &op, int64_t bound, V *part, const char *name, hipStream_t s) {
    const int64_t tiles = (bound + kScanTile - 1) / kScanTile;
    if (tiles > 0) {
        KernelTimer t(name, s);
        hipLaunchKernelGGL((k_scan_tiles<Op, V>), dim3((unsigned)tiles), dim3(kScanThreads), 0, s,
                           op, part);
    }
    {
        KernelTimer t(name, s);
        hipLaunchKernelGGL((k_scan_spine<Op, V>), dim3(1), dim3(1024), 0, s, op, part);
    }
    if (tiles > 0) {
        KernelTimer t(name, s);
        hipLaunchKernelGGL((k_scan_emit<Op, V>), dim3((unsigned)tiles), dim3(kScanThreads), 0, s,
                           op, (const V *)part);
    }
    GNNAV_HIP(hipGetLastError());
}

inline int64_t scan_parts(int64_t bound) {
    int64_t t = (bound + kScanTile - 1) / kScanTile;
    return t < 1 ? 1 : t;
}

}  // namespace gnnav
