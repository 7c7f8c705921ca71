// Internal declarations shared by the gnnav HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>
#include <string>
#include <vector>

#include "gnnav.h"

namespace gnnav {

// ------------------------------------------------------------------ errors
struct Error {
    gnnav_status status;
    std::string msg;
};

[[noreturn]] inline void fail(gnnav_status st, const std::string &msg) { throw Error{st, msg}; }

#define GNNAV_HIP(call)                                                                   \
    do {                                                                                  \
        hipError_t e_ = (call);                                                           \
        if (e_ != hipSuccess)                                                             \
            ::gnnav::fail(GNNAV_E_DEVICE, std::string(#call) + ": " + hipGetErrorString(e_)); \
    } while (0)

#define GNNAV_CHECK(cond, st, msg)                    \
    do {                                              \
        if (!(cond)) ::gnnav::fail((st), (msg));      \
    } while (0)

// Pinned host allocation (hipHostMalloc with `flags`); E_NOMEM on failure.
void host_pinned_alloc(void **p, size_t bytes, unsigned flags, const char *what);

// Waits for stream `s`; E_DEVICE if device-side work has reported a failure
// (a scan look-back wait that gave up) since the last such report.
void check_device_errors(hipStream_t s);

// Runs `body`, converting exceptions into a status and the thread's error text.
void set_last_error(const std::string &msg);
template <class F>
gnnav_status guarded(F &&body) {
    try {
        set_last_error("");
        body();
        return GNNAV_OK;
    } catch (const Error &e) {
        set_last_error(e.msg);
        return e.status;
    } catch (const std::bad_alloc &) {
        set_last_error("host allocation failed");
        return GNNAV_E_NOMEM;
    } catch (const std::exception &e) {
        set_last_error(e.what());
        return GNNAV_E_DEVICE;
    }
}

// --------------------------------------------------- grow-only device buffer
// Reallocation waits for `stream` so in-flight kernels never see a freed buffer.
struct DevBuf {
    void *p = nullptr;
    size_t bytes = 0;
    void ensure(size_t need, hipStream_t stream);
    void release();
    template <class T>
    T *as() const { return static_cast<T *>(p); }
};

// -------------------------------------------------------------- profiling
// When profiling is on, each Launch records a start/stop event pair around
// the kernel on the stream the kernel is enqueued on.
bool profiling_on();
struct KernelTimer {
    KernelTimer(const char *name, hipStream_t s);
    ~KernelTimer();
    int slot = -1;
    hipStream_t stream;
};

inline unsigned grid_for(int64_t items, int64_t per_block, int64_t cap) {
    int64_t g = (items + per_block - 1) / per_block;
    if (g > cap) g = cap;
    return (unsigned)(g < 1 ? 1 : g);
}

// ------------------------------------------------------ device primitives
constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// bf16 bit pattern of a float, round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ uint16_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

template <class V>
__device__ __forceinline__ V wave_inclusive_sum(V x) {
    const int lane = lane_id();
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        V y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive prefix sum over a block of NT threads; `scratch` holds NT/64
// values in LDS.  Returns the thread's exclusive prefix; `total` gets the
// block sum.  Must be called by every thread of the block.
template <class V, int NT>
__device__ __forceinline__ V block_exclusive_sum(V x, V *scratch, V &total) {
    constexpr int NW = NT / kWave;
    const int lane = lane_id(), wid = threadIdx.x / kWave;
    V inc = wave_inclusive_sum(x);
    if (lane == kWave - 1) scratch[wid] = inc;
    __syncthreads();
    if (wid == 0) {
        V t = lane < NW ? scratch[lane] : V(0);
        t = wave_inclusive_sum(t);
        if (lane < NW) scratch[lane] = t;
    }
    __syncthreads();
    V off = wid > 0 ? scratch[wid - 1] : V(0);
    total = scratch[NW - 1];
    __syncthreads();
    return off + inc - x;
}

// ------------------------------------------------------------ launchers
struct ScanState;   // scan.hpp: state of a one-launch device-wide scan
void launch_fill_i32(int32_t *p, int32_t v, int64_t n, hipStream_t s);

// sample.hip
struct SampleHopArgs {
    const void *row_ptr;
    bool offsets_i64;
    const int32_t *col;
    const int32_t *nodes;
    const int32_t *n_prev;   // device: |F_(h-1)|
    int32_t *indptr;         // device: |F_(h-1)|+1
    int32_t *nbrs;           // device: E_h
    int32_t *e_out;          // device: E_h (written)
    int32_t fanout;
    uint64_t rng_seed;
    uint32_t hop;            // 0-based
    int64_t rows_bound;
    ScanState *scan;
    const int32_t *bias_slot_map = nullptr;   // locality-biased selection when set
    uint32_t eta = 1;
    // optional: adjacency with each row's cached neighbours first (CSR order
    // within each class) and the per-vertex cached counts, for this slot map
    const int32_t *part_col = nullptr;
    const int32_t *part_cnt = nullptr;
    uint64_t *first_map = nullptr;           // node table: first position of each written id
    uint32_t map_tag = 0;                    // the node table tag of this sampling call
    // optional: the previous hop's relabel, run in the count scan's launch
    // (indices[p] = local id of list[p] from first_map)
    const int32_t *relabel_list = nullptr;
    const int32_t *relabel_len = nullptr;    // device length
    int64_t relabel_bound = 0;
    const int32_t *relabel_n = nullptr;      // device size of the frontier the list was merged into
    int64_t n_nodes = 0;                     // graph size (ids outside [0, n) are never looked up)
    int32_t *relabel_indices = nullptr;
    // > 0: row i's picks go to slots [i * slot_stride, (i + 1) * slot_stride)
    // of nbrs (unused slots -1) and indptr is not read; the dedup of the slot
    // list then compacts it (no count scan before the hop)
    int32_t slot_stride = 0;
};
void launch_partition_rows(const void *row_ptr, bool offsets_i64, const int32_t *col, int64_t n,
                           const int32_t *slot_map, int32_t *part_col, int32_t *part_cnt, hipStream_t s);
void launch_count_scan(const SampleHopArgs &a, hipStream_t s);
void launch_sample_hop(const SampleHopArgs &a, hipStream_t s);

struct DedupArgs {
    const int32_t *list;     // ids to union into the frontier
    int64_t len_const;       // used when len_ptr == nullptr
    const int32_t *len_ptr;  // device length
    int64_t len_bound;
    uint64_t *map;           // node table, uint64[n_nodes] (sample.hip)
    uint32_t tag;            // this sampling call's tag in it
    int64_t n_nodes;
    int32_t *nodes;
    const int32_t *base_ptr; // device |F_(h-1)| (nullptr: 0)
    int32_t *size_out;       // device |F_h|
    int32_t *err;            // device count of out-of-range ids (nullable)
    ScanState *scan;
    bool first_done = false; // first positions already in `map` (taken while writing the list)
    // optional, for the seeds (base_ptr null): hop 1's count scan folded in,
    // writing indptr (|F_0| + 1 entries) and the edge count of fanout k
    const void *count_row_ptr = nullptr;
    bool count_i64 = false;
    int32_t count_k = 0;
    int32_t *count_indptr = nullptr;
    int32_t *count_e_out = nullptr;
    int32_t *err_next = nullptr;  // the count slot of the next call, cleared by this one (nullable)
    // optional, a slot list (SampleHopArgs::slot_stride): `list` holds
    // *base_ptr rows of slot_stride slots, -1 where unused; the scan also
    // writes the used slots in order to compact_out, their row offsets to
    // indptr_out (*base_ptr + 1 entries) and their count to e_out
    int32_t slot_stride = 0;
    int32_t *compact_out = nullptr;
    int32_t *indptr_out = nullptr;
    int32_t *e_out = nullptr;
    // optional: the previous hop's relabel, run in this scan's launch
    const int32_t *relabel_list = nullptr;
    const int32_t *relabel_len = nullptr;
    int64_t relabel_bound = 0;
    const int32_t *relabel_n = nullptr;
    int32_t *relabel_indices = nullptr;
};
void launch_dedup(const DedupArgs &a, hipStream_t s);
void launch_relabel(const int32_t *list, const int32_t *len_ptr, int64_t len_bound,
                    const uint64_t *map, int64_t n_nodes, const int32_t *n_frontier, int32_t *indices,
                    hipStream_t s);

// gather.hip
struct GatherArgs {
    const int32_t *ids;
    int64_t n_ids;           // count, or its upper bound when n_ptr is set
    const int32_t *n_ptr;    // device count (nullable)
    const int32_t *slot_map;
    int64_t n_nodes;
    const void *cache;       // device [C x ld]
    const void *store;       // device-visible store [n rows] (host-mapped or HBM)
    int64_t src_ld_bytes;    // cache row stride
    int64_t store_ld_bytes;  // store row stride
    void *out;
    int64_t out_ld_bytes;
    int64_t row_bytes;       // d * elt
    int64_t *counts;         // device int64[3]
    int32_t *dev_counts;     // device int32[2]: hits, misses
    int2 *hit_list;
    int2 *miss_list;
    ScanState *scan;
    int32_t miss_wgs;        // workgroups copying misses over the host link
};
void launch_classify(const GatherArgs &a, hipStream_t s);
void launch_gather_rows(const GatherArgs &a, hipStream_t s);
void launch_matmul_bt(const float *a, int64_t lda, int64_t m, const int32_t *m_dev, int64_t k, const float *b,
                      int64_t ldb, int64_t n, float *out, int64_t ld_out, hipStream_t s, const char *label);
// Transpose of a sampled block (destination rows per source column, in
// edge order) and its column pointers; see train.hip.
struct ScanState;
struct CscWorkspace {
    DevBuf keys[2], vals[2], hist, offs, col_ptr;
    const int32_t *sorted_rows = nullptr;
    void build(const int32_t *indptr, const int32_t *indices, int64_t n_dst, const int32_t *n_dst_dev,
               const int32_t *n_edges_dev, int64_t e_bound, int64_t n_src_bound, ScanState &scan, hipStream_t s,
               const char *label);
    void release() {
        for (int k = 0; k < 2; ++k) {
            keys[k].release();
            vals[k].release();
        }
        hist.release();
        offs.release();
        col_ptr.release();
    }
};
void launch_softmax_xent(const float *z, int64_t ldz, int64_t n, const int32_t *n_dev, int64_t C,
                         const int32_t *nodes, const int32_t *labels, float *dz, int64_t lddz, float *row_loss,
                         float *loss, hipStream_t s);
void launch_aggregate_t(const CscWorkspace &csc, const int32_t *indptr, int64_t n_src, const int32_t *n_src_dev,
                        int64_t n_self, const int32_t *n_self_dev, const float *dagg, int64_t ld_dagg,
                        const float *dself, int64_t ld_dself, const float *mask, int64_t ld_mask, int64_t d,
                        float *out, int64_t ld_out, hipStream_t s, const char *label);
void launch_wgrad(const float *x_self, int64_t ld_self, const float *agg, int64_t ld_agg, int64_t m,
                  const int32_t *m_dev, int64_t d_in, const float *dz, int64_t ld_dz, int64_t d_out, DevBuf &part,
                  float *dw, float *w, float lr, hipStream_t s, const char *label);

// cache_update.hip: the cache's update policies over the ring of dynamic
// slots [lo, lo + rn), run after a gather on its lists and output.
// FIFO: ring_ptr holds two pointer words; *parity names the current one and
// flips when an update is enqueued.
void launch_fifo_update(const GatherArgs &a, int64_t lo, int64_t rn, int32_t *owner, int32_t *slot_map,
                        int32_t *ring_ptr, int *parity, void *cache, hipStream_t s);
struct LruState {
    int64_t lo, rn;
    int32_t *order;     // [rn] ring slots, least recently used first
    int32_t *part;      // [rn] the list reordered by the last batch's hits
    uint32_t *stamp;    // [rn] epoch of the last batch that hit slot lo + i
    uint32_t *ctl;      // [0] epoch of the last batch, [1] untouched count,
                        // [2] 1 while the partition is sound
    ScanState *scan;    // ensure()d for rn
};
void launch_lru_update(const GatherArgs &a, const LruState &st, int32_t *owner, int32_t *slot_map, void *cache,
                       hipStream_t s);

// spmm.hip
void launch_aggregate_mean(const int32_t *indptr, const int32_t *indices, int64_t n_dst,
                           const int32_t *n_dst_dev, const void *x, int64_t ld_x, int64_t d, bool bf16, void *out,
                           int64_t ld_out, hipStream_t s, const char *label = "aggregate_mean");

// gemm.hip
int combine_kernel_kind(int64_t m, int64_t d_out, bool bf16);   // a GNNAV_COMBINE_* value
void launch_combine(const void *self, int64_t ld_self, const void *agg, int64_t ld_agg, int64_t m,
                    const int32_t *m_dev,
                    int64_t d_in, const void *w, int64_t d_out, bool bf16, bool relu,
                    bool out_bf16, void *out, int64_t ld_out, hipStream_t s,
                    const char *label = "combine_gemm");

}  // namespace gnnav
