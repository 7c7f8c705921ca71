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
// state in parallel, in two launches: with m misses only admissions
// i >= first = max(0, m - rn) survive, into the distinct slots
// S(first .. m-1).  The admit pass gives each such slot to one lane group,
// which unmaps the slot's previous vertex where the slot map still points
// there, records the new one, copies its row, and takes the minimum of
// -3 - (i - first) over the vertex's entry in the slot map (codes below
// every slot and below -1), so among repeats of a vertex the last admitted
// one wins; the map pass lets the one admission whose code won write its
// slot, then moves the policy's starting point on.  Unmapping and
// admitting share no vertex: a vertex still mapped somewhere is a hit, not
// a miss.  The new rows are copied from the gather's output, so nothing is
// read twice over the host link.  Entries whose output row lies outside the
// request count are skipped (see k_gather_rows).
//
// FIFO keeps two ring pointer words and a parity the host flips per update:
// the map pass reads one word and writes the next pointer to the other, so
// no workgroup can see the pointer move under it.
//
// LRU's reorder is a stable partition of the list by "hit by this batch": a
// per-slot stamp set to the batch's epoch by the hits, one device-wide scan
// that writes the untouched slots to the front of `part` and the touched
// ones, reversed, to its back, and in the map pass a rotation by m that
// makes `part` the next batch's list (the admitted slots, in admission
// order, now last).  Epochs are 32-bit and stamps start at 0: a slot
// untouched for 2^32 - 1 batches would read as touched once, which only
// reorders it.  A partition scan whose look-back wait gave up may leave
// `part` with repeats, and two admissions in one slot would corrupt the
// cache; so the touch kernel raises a "partition sound" flag, a tile of the
// scan that gives up lowers it, and with the flag down the admit and map
// passes skip the batch whole: the cache stays as it was, and the next
// synchronisation point reports the failure.
#include <algorithm>

#include "common.hpp"
#include "scan.hpp"

namespace gnnav {

namespace {

// S(i) for FIFO: b = ring pointer, read from ptr[parity]; the map pass
// writes the next one to ptr[1 - parity].
struct FifoPick {
    int32_t *ptr;
    int parity;
    int64_t lo, rn;
    __device__ bool ok() const { return true; }
    __device__ int64_t base() const { return ptr[parity]; }
    __device__ int64_t slot(int64_t i, int64_t b) const { return lo + (b + i) % rn; }
    __device__ void after_map(bool, int64_t gid, int64_t, int64_t m, int64_t b) const {
        if (gid == 0) ptr[1 - parity] = (int32_t)((b + m) % rn);
    }
};

// S(i) for LRU: the reordered list is part[0 .. b) (untouched, in order)
// followed by part[rn-1], part[rn-2], ..., part[b] (touched, in order);
// b = untouched count, written by the partition scan; ok() is false when
// that scan gave up (the update is then skipped).  After the map pass the
// list becomes the reordered one rotated by m (kept as it was when the
// update was skipped), and the epoch advances.
struct LruPick {
    const int32_t *part;
    int32_t *order;
    uint32_t *ctl;   // [0] epoch, [1] untouched count, [2] 1 while the partition is sound
    int64_t rn;
    __device__ bool ok() const { return ctl[2] != 0u; }
    __device__ int64_t base() const { return (int64_t)ctl[1]; }
    __device__ int64_t slot(int64_t i, int64_t b) const {
        const int64_t j = i % rn;
        return j < b ? part[j] : part[rn - 1 - (j - b)];
    }
    __device__ void after_map(bool ok, int64_t gid, int64_t stride, int64_t m, int64_t b) const {
        if (ok)
            for (int64_t p = gid; p < rn; p += stride) order[p] = (int32_t)slot(p + m, b);
        if (gid == 0) ctl[0] += 1u;
    }
};

__device__ __forceinline__ int32_t admit_code(int64_t i, int64_t first) { return (int32_t)(-3 - (i - first)); }

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
            const int32_t u = owner[slot];
            if (u >= 0 && slot_map[u] == (int32_t)slot) slot_map[u] = -1;
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
    const bool ok = pick.ok();
    const int64_t m = *m_ptr, b = pick.base();
    if (n_ptr) n_req = *n_ptr;
    const int64_t first = m > rn ? m - rn : 0;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    if (ok) {
        for (int64_t i = first + gid; i < m; i += stride) {
            const int2 e = miss_list[i];
            if ((uint32_t)e.x >= (uint64_t)n_req) continue;
            if (slot_map[e.y] == admit_code(i, first)) slot_map[e.y] = (int32_t)pick.slot(i, b);
        }
    }
    pick.after_map(ok, gid, stride, m, b);
}

// The two passes; `map_items` sizes the map pass's grid (LRU's rotation
// covers the whole ring).
template <class Pick>
void launch_admissions(const GatherArgs &a, const Pick &pick, int64_t rn, int64_t map_items, int32_t *owner,
                       int32_t *slot_map, void *cache, hipStream_t s) {
    const int32_t *m_ptr = a.dev_counts + 1;
    const int32_t chunks = (int32_t)((a.row_bytes + 15) / 16);
    int g = 1;
    while (g < chunks && g < kWave) g <<= 1;
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
        hipLaunchKernelGGL((k_ring_map<Pick>), dim3(grid_for(map_items, 256, 4096)), dim3(256), 0, s, a.miss_list,
                           m_ptr, a.n_ptr, a.n_ids, pick, rn, slot_map);
    }
}

// LRU: stamp the ring slots this batch hit with the next epoch (ctl[0] + 1)
// and raise the "partition sound" flag for the scan that follows.
__global__ void __launch_bounds__(256) k_lru_touch(const int2 *__restrict__ hit_list,
                                                   const int32_t *__restrict__ h_ptr,
                                                   const int32_t *__restrict__ n_ptr, int64_t n_req, int64_t lo,
                                                   int64_t rn, uint32_t *__restrict__ stamp,
                                                   uint32_t *__restrict__ ctl) {
    const int64_t h = *h_ptr;
    if (n_ptr) n_req = *n_ptr;
    const uint32_t next = ctl[0] + 1u;
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl[2] = 1u;
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
    uint32_t *ctl;
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
    __device__ void gave_up() const { ctl[2] = 0u; }
};

}  // namespace

void launch_fifo_update(const GatherArgs &a, int64_t lo, int64_t rn, int32_t *owner, int32_t *slot_map,
                        int32_t *ring_ptr, int *parity, void *cache, hipStream_t s) {
    if (rn <= 0 || a.n_ids <= 0) return;
    launch_admissions(a, FifoPick{ring_ptr, *parity, lo, rn}, rn, std::min<int64_t>(a.n_ids, rn), owner, slot_map,
                      cache, s);
    *parity ^= 1;
    GNNAV_HIP(hipGetLastError());
}

void launch_lru_update(const GatherArgs &a, const LruState &st, int32_t *owner, int32_t *slot_map, void *cache,
                       hipStream_t s) {
    const int64_t rn = st.rn;
    if (rn <= 0 || a.n_ids <= 0) return;
    {
        KernelTimer t("cache_touch", s);
        hipLaunchKernelGGL(k_lru_touch, dim3(grid_for(std::min<int64_t>(a.n_ids, rn), 256, 4096)), dim3(256), 0, s,
                           a.hit_list, a.dev_counts, a.n_ptr, a.n_ids, st.lo, rn, st.stamp, st.ctl);
    }
    run_scan<LruPartitionOp, int64_t>(LruPartitionOp{st.order, st.stamp, st.ctl, st.part, st.lo, rn}, rn, *st.scan,
                                      "cache_order", s);
    launch_admissions(a, LruPick{st.part, st.order, st.ctl, rn}, rn, rn, owner, slot_map, cache, s);
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
