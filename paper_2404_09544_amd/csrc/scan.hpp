// Device-wide exclusive scan with a per-element emit step, in one launch.
//
// An Op supplies, on the device:
//   int64_t n() const                    element count (may be read from HBM)
//   V value(int64_t i) const             contribution of element i
//   void emit(int64_t i, V prefix, V v)  called for every i with its
//                                        exclusive prefix (sum over j < i)
//   void total(V t)                      called once with the grand total
// or, to read each element's inputs once for both passes, a type Item with
//   Item load(int64_t i) const, V value(const Item &) const and
//   void emit(int64_t i, V prefix, V v, const Item &) const
// (the items stay in registers between the two passes), and optionally
//   void gave_up() const                 called by a tile whose look-back
//                                        wait gave up (see below).
//
// Single-pass scan with decoupled look-back: workgroups claim tiles in order
// from an atomic ticket (so a tile only ever waits for tiles whose
// workgroups are already running) until the tiles run out; the grid is
// capped, not sized to the element bound, and workgroups beyond the tile
// count of the actual length (read on the device) leave before touching the
// ticket, so a loose bound costs an empty workgroup each, not a contended
// atomic each.  A workgroup reduces its tile,
// publishes the tile sum, then
// looks back: its first wavefront polls the 64 preceding tiles at once,
// finds the nearest one that has published an inclusive prefix, adds that
// prefix and the tile sums in between (a wave reduction), and moves the
// window back by 64 tiles if none has.  It then publishes its own inclusive
// prefix and emits.  Records carry the call's epoch, so they never need
// clearing between calls.  Each thread owns kScanItems consecutive elements,
// so results do not depend on scheduling.  The look-back wait is bounded: a
// wait that exceeds the spin limit (kSpinLimit polls unless a test lowers it)
// gives up, adds one to the library's device error word and lets the
// workgroup finish.  The prefix it publishes is then the part it had summed,
// never more than the true one, so every position derived from it stays
// inside the buffers sized for the true one; the results are wrong and the
// next synchronisation point reports E_DEVICE.
//
// Publication is one 64-bit atomic store per 32-bit half of the value, each
// word carrying the call's tag (epoch and kind) next to its half, and a
// reader takes a record only when every word shows the current tag.  No
// ordering between separate stores is needed, so publishing needs no
// release fence and reading no acquire fence: on this chip those write back
// and invalidate the whole L2 of the issuing XCD, a cost every tile would
// otherwise pay twice and that evicted the other workgroups' working sets.
#pragma once

#include <algorithm>
#include <type_traits>
#include <utility>

#include "common.hpp"

namespace gnnav {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

template <class Op, class = void>
struct ScanHasItem : std::false_type {};
template <class Op>
struct ScanHasItem<Op, std::void_t<typename Op::Item>> : std::true_type {};

template <class Op, class = void>
struct ScanHasGaveUp : std::false_type {};
template <class Op>
struct ScanHasGaveUp<Op, std::void_t<decltype(std::declval<const Op &>().gave_up())>> : std::true_type {};

template <class Op, bool = ScanHasItem<Op>::value>
struct ScanItems {   // no items: values are recomputed by index
    __device__ void load(const Op &, int, int64_t) {}
    template <class V>
    __device__ V value(const Op &op, int, int64_t i) const { return op.value(i); }
    template <class V>
    __device__ void emit(const Op &op, int, int64_t i, V prefix, V v) const { op.emit(i, prefix, v); }
};
template <class Op>
struct ScanItems<Op, true> {
    typename Op::Item it[kScanItems];
    __device__ void load(const Op &op, int j, int64_t i) { it[j] = op.load(i); }
    template <class V>
    __device__ V value(const Op &op, int j, int64_t) const { return op.value(it[j]); }
    template <class V>
    __device__ void emit(const Op &op, int j, int64_t i, V prefix, V v) const { op.emit(i, prefix, v, it[j]); }
};

constexpr uint32_t kSpinLimit = 1u << 20;
constexpr int64_t kScanGrid = 1024;   // workgroups per scan launch, at most

// Look-back polls before a wait gives up (kSpinLimit unless lowered for a
// test; 0 gives up before the first poll, so every tile after the first
// times out), and the device word that counts the waits that gave up (api.hip).
uint32_t scan_spin_limit();
uint32_t *device_error_word();

inline int64_t scan_parts(int64_t bound) {
    int64_t t = (bound + kScanTile - 1) / kScanTile;
    return t < 1 ? 1 : t;
}

// Device state of one scan sequence (calls on one stream, in order).
// Records: per tile, kRecWords words of (tag << 32 | 32-bit half of the
// value), tag = (epoch << 2) | kind, kind 1 in `sums` (the tile's own sum)
// and 2 in `prefix` (inclusive prefix through the tile).
constexpr int kRecWords = 2;   // enough for 64-bit values
struct ScanState {
    DevBuf sums;      // uint64 [tiles][kRecWords]
    DevBuf prefix;    // uint64 [tiles][kRecWords]
    DevBuf ctl;       // uint32 [0] ticket
    int64_t tiles = 0;
    uint32_t epoch = 0;
    void ensure(int64_t bound, hipStream_t s) {
        const int64_t t = scan_parts(bound);
        if (!ctl.p) {
            ctl.ensure(4 * sizeof(uint32_t), s);
            launch_fill_i32(ctl.as<int32_t>(), 0, 4, s);
        }
        if (t > tiles) {
            // a reallocation frees the old records first: until both are in
            // place and cleared no tile count may claim them
            tiles = 0;
            const size_t bytes = (size_t)t * kRecWords * sizeof(uint64_t);
            sums.ensure(bytes, s);
            prefix.ensure(bytes, s);
            tiles = (int64_t)(std::min(sums.bytes, prefix.bytes) / (kRecWords * sizeof(uint64_t)));
            launch_fill_i32(sums.as<int32_t>(), 0, tiles * kRecWords * 2, s);
            launch_fill_i32(prefix.as<int32_t>(), 0, tiles * kRecWords * 2, s);
        }
    }
    void release() {
        sums.release();
        prefix.release();
        ctl.release();
        tiles = 0;
    }
    uint32_t next_epoch() {
        epoch = (epoch + 1) & 0x3fffffffu;
        if (epoch == 0) epoch = 1;
        return epoch;
    }
};

template <class V>
__device__ __forceinline__ void publish(uint64_t *rec, int64_t tile, V v, uint32_t tag) {
    static_assert(sizeof(V) == 4 || sizeof(V) == 8, "32- or 64-bit scan values");
    const uint64_t bits = sizeof(V) == 8 ? (uint64_t)(int64_t)v : (uint64_t)(uint32_t)(int32_t)v;
    uint64_t *w = rec + tile * kRecWords;
    __hip_atomic_store(&w[0], ((uint64_t)tag << 32) | (bits & 0xffffffffull), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    if constexpr (sizeof(V) == 8)
        __hip_atomic_store(&w[1], ((uint64_t)tag << 32) | (bits >> 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The record of `tile` if every word carries `tag`.
template <class V>
__device__ __forceinline__ bool read_record(const uint64_t *rec, int64_t tile, uint32_t tag, V &v) {
    const uint64_t *w = rec + tile * kRecWords;
    const uint64_t w0 = __hip_atomic_load(&w[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((uint32_t)(w0 >> 32) != tag) return false;
    if constexpr (sizeof(V) == 8) {
        const uint64_t w1 = __hip_atomic_load(&w[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((uint32_t)(w1 >> 32) != tag) return false;
        v = (V)(int64_t)((w1 << 32) | (w0 & 0xffffffffull));
    } else {
        v = (V)(int32_t)(uint32_t)w0;
    }
    return true;
}

// An element-wise job that rides along in a scan's launch (Side::n() items,
// Side::run(i) for each) on workgroups of its own: independent work that
// would otherwise cost a launch of its own.
struct NoSide {
    __device__ int64_t n() const { return 0; }
    __device__ void run(int64_t) const {}
};

template <class Op, class V, class Side>
__global__ void __launch_bounds__(kScanThreads) k_scan_onepass(Op op, Side side, int scan_grid,
                                                                uint64_t *__restrict__ sums,
                                                                uint64_t *__restrict__ prefix,
                                                                uint32_t *__restrict__ ctl, uint32_t epoch,
                                                                uint32_t *__restrict__ errors, uint32_t spin_limit) {
    __shared__ V scratch[kScanThreads / kWave];
    __shared__ int64_t s_tile;
    __shared__ V s_prefix;
    if ((int)blockIdx.x >= scan_grid) {   // the side job's workgroups
        const int64_t m = side.n(), stride = (int64_t)(gridDim.x - scan_grid) * kScanThreads;
        for (int64_t i = (int64_t)(blockIdx.x - scan_grid) * kScanThreads + threadIdx.x; i < m; i += stride)
            side.run(i);
        return;
    }
    const int64_t n = op.n();
    int64_t ntiles = (n + kScanTile - 1) / kScanTile;
    if (ntiles < 1) ntiles = 1;
    const int64_t workers = ntiles < (int64_t)scan_grid ? ntiles : (int64_t)scan_grid;
    if ((int64_t)blockIdx.x >= workers) return;
    for (;;) {
        // Every worker draws tickets until it draws one past the last tile,
        // so exactly ntiles + workers tickets are drawn per launch; the
        // workgroup that draws the final one resets the counter for the next.
        if (threadIdx.x == 0) {
            const uint32_t t = atomicAdd(&ctl[0], 1u);
            if ((int64_t)t == ntiles + workers - 1) atomicExch(&ctl[0], 0u);
            s_tile = t;
        }
        __syncthreads();
        const int64_t tile = s_tile;
        if (tile >= ntiles) return;   // uniform across the workgroup

        const int64_t first = tile * kScanTile + (int64_t)threadIdx.x * kScanItems;
        V vals[kScanItems];
        ScanItems<Op> items;
        V s = V(0);
    #pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int64_t i = first + j;
            if (i < n) items.load(op, j, i);
        }
    #pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int64_t i = first + j;
            vals[j] = i < n ? items.template value<V>(op, j, i) : V(0);
            s += vals[j];
        }
        V total;
        const V ex = block_exclusive_sum<V, kScanThreads>(s, scratch, total);

        if (threadIdx.x < kWave) {
            const int lane = threadIdx.x;
            const uint32_t tag = epoch << 2;
            V pre = V(0);
            if (tile == 0) {
                if (lane == 0) publish(prefix, 0, total, tag | 2u);
            } else {
                if (lane == 0) publish(sums, tile, total, tag | 1u);
                int64_t base = tile - 1;
                uint32_t spins = 0;
                while (true) {
                    if (spins >= spin_limit) {
                        if (lane == 0) {
                            atomicAdd(errors, 1u);
                            if constexpr (ScanHasGaveUp<Op>::value) op.gave_up();
                        }
                        break;
                    }
                    const int64_t t = base - lane;
                    // tiles before tile 0 read as a published zero prefix; the
                    // window that reaches tile 0 always stops there first
                    V v = V(0);
                    bool is_prefix = t < 0, ready = t < 0;
                    if (t >= 0) {
                        is_prefix = read_record<V>(prefix, t, tag | 2u, v);
                        ready = is_prefix || read_record<V>(sums, t, tag | 1u, v);
                    }
                    const uint64_t pmask = __ballot(is_prefix);
                    const int pidx = pmask ? __builtin_ctzll(pmask) : kWave;
                    const uint64_t need = pidx >= kWave - 1 ? ~0ull : ((1ull << (pidx + 1)) - 1);
                    if ((__ballot(ready) & need) != need) {
                        ++spins;
                        __builtin_amdgcn_s_sleep(1);
                        continue;
                    }
                    if (lane > pidx) v = V(0);
    #pragma unroll
                    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
                    pre += v;
                    if (pidx < kWave) break;
                    base -= kWave;
                    spins = 0;
                }
                if (lane == 0) publish(prefix, tile, pre + total, tag | 2u);
            }
            if (lane == 0) {
                s_prefix = pre;
                if (tile == ntiles - 1) op.total(pre + total);
            }
        }
        __syncthreads();
        V run = ex + s_prefix;
    #pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int64_t i = first + j;
            if (i < n) items.emit(op, j, i, run, vals[j]);
            run += vals[j];
        }
        __syncthreads();   // s_tile / s_prefix are reused by the next ticket
    }
}

// Enqueue one scan, and with it the side job over at most side_bound items.
// `bound` >= op.n() sizes the grid; `st` must have been ensure()d for
// `bound` on this stream.
template <class Op, class V, class Side = NoSide>
void run_scan(const Op &op, int64_t bound, ScanState &st, const char *name, hipStream_t s,
              const Side &side = Side(), int64_t side_bound = 0) {
    int64_t grid = scan_parts(bound);
    if (grid > kScanGrid) grid = kScanGrid;
    const int64_t side_grid = side_bound > 0 ? (int64_t)grid_for(side_bound, kScanThreads, 2048) : 0;
    const uint32_t epoch = st.next_epoch();
    KernelTimer t(name, s);
    hipLaunchKernelGGL((k_scan_onepass<Op, V, Side>), dim3((unsigned)(grid + side_grid)), dim3(kScanThreads), 0, s,
                       op, side, (int)grid, st.sums.as<uint64_t>(), st.prefix.as<uint64_t>(),
                       st.ctl.as<uint32_t>(), epoch, device_error_word(), scan_spin_limit());
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
