// Feature gather through the static device cache (the cache step of the
// paper's transmission abstraction: find the cached part of the batch, fetch
// the rest from the host).
//
//   classify   slot lookup per requested id; an order-preserving scan
//              splits the requests into a hit list (out row, cache slot)
//              and a miss list (out row, node id) and writes the counts;
//              out-of-range ids get a zero row right here
//   rows       copies listed rows in 16-byte units in one launch: a fixed
//              share of the workgroups reads the miss rows from the host
//              store through its device mapping (zero-copy over the host
//              link), the rest read the hit rows from the HBM cache
#include <algorithm>

#include "common.hpp"
#include "scan.hpp"

namespace gnnav {

struct ClassifyOp {
    const int32_t *ids;
    int64_t n_ids;
    const int32_t *n_ptr;
    const int32_t *slot_map;
    int64_t n_nodes;
    int2 *hit_list;
    int2 *miss_list;
    int64_t *counts;
    int32_t *dev_counts;
    uint4 *out;
    int64_t out_ld16;
    int64_t chunks;
    // the request and its slot, read once for both scan passes (slot -2:
    // id out of range)
    struct Item {
        int32_t id, slot;
    };
    // packed value: hits in the high 32 bits, misses in the low 32 bits
    __device__ int64_t n() const { return n_ptr ? (int64_t)*n_ptr : n_ids; }
    __device__ Item load(int64_t i) const {
        const int32_t id = ids[i];
        return Item{id, (id < 0 || id >= n_nodes) ? -2 : slot_map[id]};
    }
    __device__ int64_t value(const Item &it) const {
        if (it.slot == -2) return 0;
        return it.slot >= 0 ? (int64_t(1) << 32) : int64_t(1);
    }
    __device__ void emit(int64_t i, int64_t prefix, int64_t v, const Item &it) const {
        if (v == 0) {
            uint4 *row = out + i * out_ld16;
            for (int64_t c = 0; c < chunks; ++c) row[c] = make_uint4(0, 0, 0, 0);
        } else if (v == 1) {
            miss_list[(int32_t)(prefix & 0xffffffff)] = make_int2((int32_t)i, it.id);
        } else {
            hit_list[(int32_t)(prefix >> 32)] = make_int2((int32_t)i, it.slot);
        }
    }
    __device__ void total(int64_t t) const {
        const int64_t hits = t >> 32, misses = t & 0xffffffff;
        counts[0] = hits;
        counts[1] = misses;
        counts[2] = n() - hits - misses;
        dev_counts[0] = (int32_t)hits;
        dev_counts[1] = (int32_t)misses;
    }
};

void launch_classify(const GatherArgs &a, hipStream_t s) {
    ClassifyOp op{a.ids, a.n_ids, a.n_ptr, a.slot_map, a.n_nodes, a.hit_list, a.miss_list, a.counts,
                  a.dev_counts, (uint4 *)a.out, a.out_ld_bytes / 16, (a.row_bytes + 15) / 16};
    run_scan<ClassifyOp, int64_t>(op, a.n_ids, *a.scan, "classify", s);
}

// One launch moves both lists.  Workgroups [0, miss_blocks) copy the miss
// list from the host store (zero-copy over the host link), the others copy
// the hit list from the HBM cache, so the two proceed together without a
// second stream (a second stream would share one of the process's few
// hardware queues with other work and hold it for the whole transfer).
// G lanes per row (power of two), 64/G rows per wavefront pass; lane c0
// moves 16-byte units c0, c0 + G, ... of its row.  For rows of at most 512
// bytes (G < 64) a miss lane group keeps 4 rows in flight, each row's units
// loaded before any is stored: a zero-copy read waits microseconds, so short
// rows need several outstanding per lane (400-byte rows: 41.6 -> 43.7 GB/s).
// Longer rows already keep several units per lane in flight, and more rows
// at once measured slower (2.4 KB rows: 55.9 -> 55.1 GB/s with 4, and the
// pipelined step slower still); hits copy one row at a time (four rows in
// flight measured 90 -> 170 us for 99.6k 2.4 KB rows from HBM).
// A list entry whose output row lies outside the request count is skipped:
// only a classification whose scan gave up (reported as a device error) can
// leave such an entry, a stale one of an earlier call, and the output
// buffer may be shorter now.
template <int G, int U>
__device__ __forceinline__ void copy_rows(const int2 *__restrict__ list, int64_t count, int64_t first, int64_t step,
                                          int64_t n_req, const uint4 *__restrict__ src_base, int64_t src_ld16,
                                          uint4 *__restrict__ out, int64_t out_ld16, int32_t chunks, int c0) {
    for (int64_t r0 = first; r0 < count; r0 += U * step) {
        const uint4 *src[U];
        uint4 *dst[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t r = r0 + u * step;
            int2 e = make_int2(-1, 0);
            if (r < count) e = list[r];
            ok[u] = (uint32_t)e.x < (uint64_t)n_req;
            src[u] = src_base + (int64_t)(ok[u] ? e.y : 0) * src_ld16;
            dst[u] = out + (int64_t)(ok[u] ? e.x : 0) * out_ld16;
        }
        if (U > 1 && chunks <= 4 * G) {
            uint4 v[U][4];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (ok[u] && c0 + q * G < chunks) v[u][q] = src[u][c0 + q * G];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (ok[u] && c0 + q * G < chunks) dst[u][c0 + q * G] = v[u][q];
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!ok[u]) continue;
                int c = c0;
                for (; c + 3 * G < chunks; c += 4 * G) {
                    const uint4 a = src[u][c], b = src[u][c + G], x = src[u][c + 2 * G], y = src[u][c + 3 * G];
                    dst[u][c] = a;
                    dst[u][c + G] = b;
                    dst[u][c + 2 * G] = x;
                    dst[u][c + 3 * G] = y;
                }
                for (; c < chunks; c += G) dst[u][c] = src[u][c];
            }
        }
    }
}

template <int G>
__global__ void __launch_bounds__(256) k_gather_rows(const int2 *__restrict__ hit_list,
                                                     const int2 *__restrict__ miss_list,
                                                     const int32_t *__restrict__ dev_counts,
                                                     const int32_t *__restrict__ n_ptr, int64_t n_req,
                                                     const uint4 *__restrict__ cache, int64_t cache_ld16,
                                                     const uint4 *__restrict__ store, int64_t store_ld16,
                                                     uint4 *__restrict__ out, int64_t out_ld16,
                                                     int32_t chunks, int32_t miss_blocks) {
    constexpr int RPW = kWave / G;
    const int lane = lane_id();
    const int sub = lane / G, c0 = lane % G;
    const bool miss = (int32_t)blockIdx.x < miss_blocks;
    if (n_ptr) n_req = *n_ptr;
    const int64_t block = miss ? blockIdx.x : blockIdx.x - miss_blocks;
    const int64_t nblocks = miss ? miss_blocks : gridDim.x - miss_blocks;
    const int64_t nwaves = nblocks * (blockDim.x / kWave);
    const int64_t first = ((block * blockDim.x + threadIdx.x) / kWave) * RPW + sub, step = nwaves * RPW;
    if (miss)
        copy_rows<G, (G < kWave ? 4 : 1)>(miss_list, dev_counts[1], first, step, n_req, store, store_ld16, out,
                                          out_ld16, chunks, c0);
    else
        copy_rows<G, 1>(hit_list, dev_counts[0], first, step, n_req, cache, cache_ld16, out, out_ld16, chunks, c0);
}

void launch_gather_rows(const GatherArgs &a, hipStream_t s) {
    const int32_t chunks = (int32_t)((a.row_bytes + 15) / 16);
    int g = 1;
    while (g < chunks && g < kWave) g <<= 1;
    const int64_t rows_bound = a.n_ids;
    if (rows_bound <= 0 || chunks <= 0) return;
    const int rows_per_block = (256 / kWave) * (kWave / g);
    // The miss share needs only enough waves to cover the host link's
    // latency; more of them queue slow host reads in the memory system,
    // which stalls the HBM copy of the hits and any concurrent kernel.
    const unsigned miss_blocks = grid_for(rows_bound, rows_per_block, a.miss_wgs);
    const unsigned hit_blocks = grid_for(rows_bound, rows_per_block, 8192);
    const int64_t cld = a.src_ld_bytes / 16, sld = a.store_ld_bytes / 16, old = a.out_ld_bytes / 16;
    KernelTimer t("gather_rows", s);
    switch (g) {
#define GNNAV_G(GV)                                                                                       \
    case GV:                                                                                              \
        hipLaunchKernelGGL(k_gather_rows<GV>, dim3(miss_blocks + hit_blocks), dim3(256), 0, s, a.hit_list,  \
                           a.miss_list, a.dev_counts, a.n_ptr, a.n_ids, (const uint4 *)a.cache, cld,        \
                           (const uint4 *)a.store, sld,                                                     \
                           (uint4 *)a.out, old, chunks, (int32_t)miss_blocks);                             \
        break;
        GNNAV_G(1) GNNAV_G(2) GNNAV_G(4) GNNAV_G(8) GNNAV_G(16) GNNAV_G(32) GNNAV_G(64)
#undef GNNAV_G
        default:
            fail(GNNAV_E_INVALID, "bad row width");
    }
    GNNAV_HIP(hipGetLastError());
}

}  // namespace gnnav
