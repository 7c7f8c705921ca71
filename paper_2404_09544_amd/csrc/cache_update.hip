// Cache update after a gather (the cache's update policy of Section 3.2,
// "Transmission strategies"; its cost is Eq. 5's t_replace).  A policy owns
// the ring of dynamic slots [lo, lo + rn) at the end of the cache; the
// slots before it keep the degree-ranked vertices.
//
//   FIFO  the batch's misses, in request order, take the ring's slots in
//         turn from a ring pointer.
//   LRU   the ring keeps a recency list (least recent first).  The ring
//         slots the batch hit move to the back, after the untouched ones,
//         each group in its earlier order (every request of a batch is a use
//         at the same time); then the misses, in request order, take the
//         slots from the front, each becoming the most recent.
//
// Either way the i-th miss (0-based) is admitted into slot S(i): the slot
// that sits i places (mod rn) after the policy's starting point (FIFO: the
// ring pointer; LRU: the front of the reordered list).  Admitting one by
// one, as the definition does, a slot's previous vertex is evicted
// (unmapped if the slot map still points at that slot; a vertex requested
// twice in one batch is admitted twice and keeps its later slot, its
// earlier one holding a stale copy until it is evicted).  The same final
// state in parallel: with m misses only admissions i >= first =
// max(0, m - rn) survive, into the distinct slots S(first .. m-1); those
// slots are evicted (unmapped where still mapped), each takes its miss, and
// among repeats of a vertex the last admitted one is mapped: the admit pass
// takes the minimum of -3 - (i - first) per vertex in the slot map (codes
// below every slot and below -1), the map pass lets the one admission whose
// code won write its slot.  The new rows are copied from the gather's
// output, so nothing is read twice over the host link.  Entries whose
// output row lies outside the request count are skipped (see
// k_gather_rows).
//
// LRU's reorder is a stable partition of the list by "hit by this batch": a
// per-slot stamp set to the batch's epoch by the hits, one device-wide scan
// that writes the untouched slots to the front of `part` and the touched
// ones, reversed, to its back, and after the admissions a rotation by m
// that makes `part` the next batch's list (the admitted slots, in
// admission order, now last).  Epochs are 32-bit and stamps start at 0: a
// slot untouched for 2^32 - 1 batches would read as touched once, which
// only reorders it.  A partition scan whose look-back wait gave up may leave
// `part` with repeats, and two admissions in one slot would corrupt the
// cache; so the device error word (which only grows) is read before and
// after the scan, one thread records whether it moved, and if it did the
// update is skipped as a whole: the cache stays as it was, and the next
// synchronisation point reports the failure.
#include <algorithm>

#include "common.hpp"
#include "scan.hpp"

namespace gnnav {

namespace {

// S(i) for FIFO: b = ring pointer.
struct FifoPick {
    const int32_t *ring_ptr;
    int64_t lo, rn;
    __device__ bool ok() const { return true; }
    __device__ int64_t base() const { return *ring_ptr; }
    __device__ int64_t slot(int64_t i, int64_t b) const { return lo + (b + i) % rn; }
};

// S(i) for LRU: the reordered list is part[0 .. b) (untouched, in order)
// followed by part[rn-1], part[rn-2], ..., part[b] (touched, in order);
// b = untouched count, written by the partition scan; ok() is false when
// that scan gave up (the update is then skipped).
struct LruPick {
    const int32_t *part;
    const uint32_t *ctl;   // [1] untouched count, [3] 1 if the partition is sound
    int64_t rn;
    __device__ bool ok() const { return ctl[3] != 0u; }
    __device__ int64_t base() const { return (int64_t)ctl[1]; }
    __device__ int64_t slot(int64_t i, int64_t b) const {
        const int64_t j = i % rn;
        return j < b ? part[j] : part[rn - 1 - (j - b)];
    }
};

__device__ __forceinline__ int32_t admit_code(int64_t i, int64_t first) { return (int32_t)(-3 - (i - first)); }

template <class Pick>
__global__ void __launch_bounds__(256) k_ring_evict(const int32_t *__restrict__ m_ptr, Pick pick, int64_t rn,
                                                    const int32_t *__restrict__ owner,
                                                    int32_t *__restrict__ slot_map) {
    if (!pick.ok()) return;
    const int64_t m = *m_ptr, b = pick.base();
    const int64_t first = m > rn ? m - rn : 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = first + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        const int64_t slot = pick.slot(i, b);
        const int32_t v = owner[slot];
        if (v >= 0 && slot_map[v] == (int32_t)slot) slot_map[v] = -1;
    }
}

template <int G, class Pick>
__global__ void __launch_bounds__(256) k_ring_admit(const int2 *__restrict__ miss_list,
                                                    const int32_t *__restrict__ m_ptr,
                                                    const int32_t *__restrict__ n_ptr, int64_t n_req, Pick pick,
                                                    int64_t rn, int32_t *__restrict__ owner,
                                                    int32_t *__restrict__ slot_map, const uint4 *__restrict__ out,
                                                    int64_t out_ld16, uint4 *__restrict__ cache, int64_t cache_ld16,
                                                    int32_t chunks) {
    constexpr int RPW = kWave / G;
    if (!pick.ok()) return;
    const int lane = lane_id();
    const int sub = lane / G, c0 = lane % G;
    const int64_t m = *m_ptr, b = pick.base();
    if (n_ptr) n_req = *n_ptr;
    const int64_t first = m > rn ? m - rn : 0;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / kWave;
    for (int64_t i = first + (((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave) * RPW + sub; i < m;
         i += nwaves * RPW) {
        const int2 e = miss_list[i];
        if ((uint32_t)e.x >= (uint64_t)n_req) continue;
        const int64_t slot = pick.slot(i, b);
        if (c0 == 0) {
            owner[slot] = e.y;
            atomicMin(&slot_map[e.y], admit_code(i, first));
        }
        const uint4 *src = out + (int64_t)e.x * out_ld16;
        uint4 *dst = cache + slot * cache_ld16;
        for (int c = c0; c < chunks; c += G) dst[c] = src[c];
    }
}

template <class Pick>
__global__ void __launch_bounds__(256) k_ring_map(const int2 *__restrict__ miss_list,
                                                  const int32_t *__restrict__ m_ptr,
                                                  const int32_t *__restrict__ n_ptr, int64_t n_req, Pick pick,
                                                  int64_t rn, int32_t *__restrict__ slot_map) {
    if (!pick.ok()) return;
    const int64_t m = *m_ptr, b = pick.base();
    if (n_ptr) n_req = *n_ptr;
    const int64_t first = m > rn ? m - rn : 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = first + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        const int2 e = miss_list[i];
        if ((uint32_t)e.x >= (uint64_t)n_req) continue;
        if (slot_map[e.y] == admit_code(i, first)) slot_map[e.y] = (int32_t)pick.slot(i, b);
    }
}

template <class Pick>
void launch_admissions(const GatherArgs &a, const Pick &pick, int64_t rn, int32_t *owner, int32_t *slot_map,
                       void *cache, hipStream_t s) {
    const int32_t *m_ptr = a.dev_counts + 1;
    const int32_t chunks = (int32_t)((a.row_bytes + 15) / 16);
    int g = 1;
    while (g < chunks && g < kWave) g <<= 1;
    const unsigned grid1 = grid_for(std::min<int64_t>(a.n_ids, rn), 256, 4096);
    {
        KernelTimer t("cache_evict", s);
        hipLaunchKernelGGL((k_ring_evict<Pick>), dim3(grid1), dim3(256), 0, s, m_ptr, pick, rn, owner, slot_map);
    }
    {
        KernelTimer t("cache_admit", s);
        const unsigned grid = grid_for(std::min<int64_t>(a.n_ids, rn), (256 / kWave) * (kWave / g), 4096);
        switch (g) {
#define GNNAV_G(GV)                                                                                          \
    case GV:                                                                                                 \
        hipLaunchKernelGGL((k_ring_admit<GV, Pick>), dim3(grid), dim3(256), 0, s, a.miss_list, m_ptr, a.n_ptr,  \
                           a.n_ids, pick, rn, owner, slot_map, (const uint4 *)a.out, a.out_ld_bytes / 16,      \
                           (uint4 *)cache, a.src_ld_bytes / 16, chunks);                                       \
        break;
            GNNAV_G(1) GNNAV_G(2) GNNAV_G(4) GNNAV_G(8) GNNAV_G(16) GNNAV_G(32) GNNAV_G(64)
#undef GNNAV_G
            default:
                fail(GNNAV_E_INVALID, "bad row width");
        }
    }
    {
        KernelTimer t("cache_map", s);
        hipLaunchKernelGGL((k_ring_map<Pick>), dim3(grid1), dim3(256), 0, s, a.miss_list, m_ptr, a.n_ptr, a.n_ids,
                           pick, rn, slot_map);
    }
}

__global__ void k_fifo_advance(const int32_t *__restrict__ m_ptr, int32_t *__restrict__ ring_ptr, int64_t rn) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *ring_ptr = (int32_t)(((int64_t)*ring_ptr + *m_ptr) % rn);
}

__device__ __forceinline__ uint32_t error_count(const uint32_t *err) {
    return __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// LRU: stamp the ring slots this batch hit with the next epoch (ctl[0] + 1);
// record the device error count (ctl[2]) before the partition scan.
__global__ void __launch_bounds__(256) k_lru_touch(const int2 *__restrict__ hit_list,
                                                   const int32_t *__restrict__ h_ptr,
                                                   const int32_t *__restrict__ n_ptr, int64_t n_req, int64_t lo,
                                                   int64_t rn, uint32_t *__restrict__ stamp,
                                                   uint32_t *__restrict__ ctl, const uint32_t *__restrict__ err) {
    const int64_t h = *h_ptr;
    if (n_ptr) n_req = *n_ptr;
    const uint32_t next = ctl[0] + 1u;
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl[2] = error_count(err);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < h; i += stride) {
        const int2 e = hit_list[i];
        if ((uint32_t)e.x >= (uint64_t)n_req) continue;
        const int64_t r = (int64_t)e.y - lo;
        if (r >= 0 && r < rn) stamp[r] = next;
    }
}

// LRU: stable partition of the recency list by the stamps.  Packed value:
// touched in the high 32 bits, untouched in the low 32 bits.
struct LruPartitionOp {
    const int32_t *order;
    const uint32_t *stamp;
    uint32_t *ctl;      // [0] epoch of the last batch, [1] untouched count
    int32_t *part;
    int64_t lo, rn;
    struct Item {
        int32_t slot;
        bool touched;
    };
    __device__ int64_t n() const { return rn; }
    __device__ Item load(int64_t i) const {
        const int32_t s = order[i];
        return Item{s, stamp[s - lo] == ctl[0] + 1u};
    }
    __device__ int64_t value(const Item &it) const { return it.touched ? (int64_t(1) << 32) : int64_t(1); }
    __device__ void emit(int64_t, int64_t prefix, int64_t, const Item &it) const {
        if (it.touched)
            part[rn - 1 - (prefix >> 32)] = it.slot;
        else
            part[prefix & 0xffffffff] = it.slot;
    }
    __device__ void total(int64_t t) const { ctl[1] = (uint32_t)(t & 0xffffffff); }
};

// LRU: ctl[3] = 1 if no look-back wait gave up since the touch kernel ran.
__global__ void k_lru_check(uint32_t *__restrict__ ctl, const uint32_t *__restrict__ err) {
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl[3] = error_count(err) == ctl[2] ? 1u : 0u;
}

// LRU: the next batch's list is the reordered one rotated by m (the slots
// S(0 .. m-1) were used last, in admission order; kept as it was when the
// update was skipped); then the epoch advances.
__global__ void __launch_bounds__(256) k_lru_rotate(LruPick pick, const int32_t *__restrict__ m_ptr,
                                                    int32_t *__restrict__ order, uint32_t *__restrict__ ctl) {
    if (pick.ok()) {
        const int64_t m = *m_ptr, b = pick.base();
        const int64_t stride = (int64_t)gridDim.x * blockDim.x;
        for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < pick.rn; p += stride)
            order[p] = (int32_t)pick.slot(p + m, b);
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl[0] += 1u;
}

}  // namespace

void launch_fifo_update(const GatherArgs &a, int64_t lo, int64_t rn, int32_t *owner, int32_t *slot_map,
                        int32_t *ring_ptr, void *cache, hipStream_t s) {
    if (rn <= 0 || a.n_ids <= 0) return;
    launch_admissions(a, FifoPick{ring_ptr, lo, rn}, rn, owner, slot_map, cache, s);
    {
        KernelTimer t("cache_advance", s);
        hipLaunchKernelGGL(k_fifo_advance, dim3(1), dim3(64), 0, s, a.dev_counts + 1, ring_ptr, rn);
    }
    GNNAV_HIP(hipGetLastError());
}

void launch_lru_update(const GatherArgs &a, const LruState &st, int32_t *owner, int32_t *slot_map, void *cache,
                       hipStream_t s) {
    const int64_t rn = st.rn;
    if (rn <= 0 || a.n_ids <= 0) return;
    {
        KernelTimer t("cache_touch", s);
        hipLaunchKernelGGL(k_lru_touch, dim3(grid_for(std::min<int64_t>(a.n_ids, rn), 256, 4096)), dim3(256), 0, s,
                           a.hit_list, a.dev_counts, a.n_ptr, a.n_ids, st.lo, rn, st.stamp, st.ctl,
                           device_error_word());
    }
    run_scan<LruPartitionOp, int64_t>(LruPartitionOp{st.order, st.stamp, st.ctl, st.part, st.lo, rn}, rn, *st.scan,
                                      "cache_order", s);
    {
        KernelTimer t("cache_check", s);
        hipLaunchKernelGGL(k_lru_check, dim3(1), dim3(64), 0, s, st.ctl, (const uint32_t *)device_error_word());
    }
    const LruPick pick{st.part, st.ctl, rn};
    launch_admissions(a, pick, rn, owner, slot_map, cache, s);
    {
        KernelTimer t("cache_rotate", s);
        hipLaunchKernelGGL(k_lru_rotate, dim3(grid_for(rn, 256, 2048)), dim3(256), 0, s, pick, a.dev_counts + 1,
                           st.order, st.ctl);
    }
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
