// C ABI of the sampled mini-batch step (declarations and contracts in
// include/gnnav.h): handles, argument checks, one-time set-up on the host
// (CSR build, degree ranking, pinned store), and the per-batch
// orchestration that enqueues the kernels of sample.hip, gather.hip,
// spmm.hip and gemm.hip.
#include <algorithm>
#include <atomic>
#include <functional>
#include <cmath>
#include <cstring>
#include <mutex>
#include <thread>

#include "common.hpp"
#include "scan.hpp"

using namespace gnnav;

// ------------------------------------------------------------------ errors
namespace gnnav {
static thread_local std::string t_last_error;
void set_last_error(const std::string &msg) { t_last_error = msg; }
}  // namespace gnnav

extern "C" const char *gnnav_last_error(void) { return t_last_error.c_str(); }
extern "C" int32_t gnnav_abi_version(void) { return GNNAV_ABI_VERSION; }

// ------------------------------------------------- allocation-failure hook
// Testing aid (gnnav_debug_fail_allocations): after `g_alloc_budget` more
// successful device or pinned allocations, every further one fails as if the
// memory were exhausted.  Negative: off.
namespace {
std::atomic<int64_t> g_alloc_budget{-1};
bool alloc_denied() {
    int64_t b = g_alloc_budget.load();
    while (b >= 0) {
        if (b == 0) return true;
        if (g_alloc_budget.compare_exchange_weak(b, b - 1)) return false;
    }
    return false;
}
}  // namespace

namespace gnnav {
void host_pinned_alloc(void **p, size_t bytes, unsigned flags, const char *what) {
    *p = nullptr;
    if (alloc_denied() || hipHostMalloc(p, bytes, flags) != hipSuccess) {
        (void)hipGetLastError();
        *p = nullptr;
        fail(GNNAV_E_NOMEM, std::string("pinned host allocation of ") + std::to_string(bytes) + " bytes (" + what +
                                ") failed");
    }
}
}  // namespace gnnav

extern "C" gnnav_status gnnav_debug_fail_allocations(int64_t after) {
    g_alloc_budget.store(after < 0 ? -1 : after);
    return GNNAV_OK;
}

// ---------------------------------------------------------- device buffer
void DevBuf::ensure(size_t need, hipStream_t stream) {
    if (need <= bytes && p) return;
    if (p) {
        GNNAV_HIP(hipStreamSynchronize(stream));
        GNNAV_HIP(hipFree(p));
        p = nullptr;
        bytes = 0;
    }
    size_t b = need < 256 ? 256 : need;
    b += b / 8;  // headroom so slowly growing batches do not reallocate every time
    if (alloc_denied() || hipMalloc(&p, b) != hipSuccess) {
        (void)hipGetLastError();
        p = nullptr;
        fail(GNNAV_E_NOMEM, "device allocation of " + std::to_string(b) + " bytes failed");
    }
    bytes = b;
}

// ----------------------------------------------------- device error word
// One word per device, counting the device-wide scans' look-back waits that
// gave up (see scan.hpp).  It only grows; each synchronisation point compares
// it with the count already reported on that device, so a failure of any
// asynchronous work is reported once, by the first synchronisation point that
// follows it.  A static device variable: nothing is allocated for it.
static __device__ uint32_t g_device_errors;

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_err_mu;
uint32_t *g_err_ptr[kMaxDevices] = {};
uint32_t g_err_seen[kMaxDevices] = {};
std::atomic<uint32_t> g_spin_limit{kSpinLimit};

int current_device() {
    int dev = 0;
    GNNAV_HIP(hipGetDevice(&dev));
    GNNAV_CHECK(dev >= 0 && dev < kMaxDevices, GNNAV_E_DEVICE, "device index beyond the library's table");
    return dev;
}
}  // namespace

namespace gnnav {
uint32_t scan_spin_limit() { return g_spin_limit.load(); }

uint32_t *device_error_word() {
    const int dev = current_device();
    std::lock_guard<std::mutex> lk(g_err_mu);
    if (!g_err_ptr[dev]) {
        void *ptr = nullptr;
        GNNAV_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(g_device_errors)));
        g_err_ptr[dev] = (uint32_t *)ptr;
    }
    return g_err_ptr[dev];
}

// Waits for `s`, then fails with E_DEVICE if the current device's error word
// has grown since it was last reported.
void check_device_errors(hipStream_t s) {
    uint32_t *w = device_error_word();
    uint32_t now = 0;
    GNNAV_HIP(hipMemcpyAsync(&now, w, sizeof(now), hipMemcpyDeviceToHost, s));
    GNNAV_HIP(hipStreamSynchronize(s));
    const int dev = current_device();
    uint32_t fresh;
    {
        std::lock_guard<std::mutex> lk(g_err_mu);
        fresh = now - g_err_seen[dev];
        g_err_seen[dev] = now;
    }
    GNNAV_CHECK(fresh == 0, GNNAV_E_DEVICE,
                std::to_string(fresh) + " device-wide scan look-back wait(s) gave up; results of the work "
                "enqueued since the last synchronisation point are unreliable");
}
}  // namespace gnnav

extern "C" gnnav_status gnnav_sync(void *stream) {
    return guarded([&] { check_device_errors((hipStream_t)stream); });
}

// Share `part` of `parts`: CU-mask bits i with (i / 8) % parts == part.  The
// runtime deals mask bits out to the eight XCDs in turn (bit i drives unit
// i / 8 of XCD i % 8, read back from the XCC and HW_ID registers of the
// workgroups of masked streams), so each share holds every parts-th unit of
// every XCD; with two shares, two of the four shader engines of each XCD.
extern "C" gnnav_status gnnav_stream_create(int32_t part, int32_t parts, void **out) {
    return guarded([&] {
        GNNAV_CHECK(out, GNNAV_E_INVALID, "out is NULL");
        GNNAV_CHECK(parts >= 1 && parts <= 8, GNNAV_E_INVALID, "parts outside [1, 8]");
        GNNAV_CHECK(part >= 0 && part < parts, GNNAV_E_INVALID, "part outside [0, parts)");
        int n_cu = 0;
        GNNAV_HIP(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, current_device()));
        GNNAV_CHECK(n_cu >= 8 * parts, GNNAV_E_INVALID, "fewer than 8 compute units per share");
        std::vector<uint32_t> mask((size_t)(n_cu + 31) / 32, 0u);
        for (int i = 0; i < n_cu; ++i)
            if ((i / 8) % parts == part) mask[(size_t)i / 32] |= 1u << (i % 32);
        hipStream_t s = nullptr;
        GNNAV_HIP(hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data()));
        *out = (void *)s;
    });
}

extern "C" gnnav_status gnnav_stream_destroy(void *stream) {
    return guarded([&] {
        if (!stream) return;
        GNNAV_HIP(hipStreamSynchronize((hipStream_t)stream));
        GNNAV_HIP(hipStreamDestroy((hipStream_t)stream));
    });
}

extern "C" gnnav_status gnnav_debug_set_spin_limit(uint32_t polls) {
    g_spin_limit.store(polls);
    return GNNAV_OK;
}
void DevBuf::release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    bytes = 0;
}

// -------------------------------------------------------------- profiling
namespace {
struct ProfEntry {
    std::string name;
    int64_t launches = 0;
    double ms = 0;
    std::vector<float> samples;   // per-launch durations, in launch order
};
struct Pending {
    int slot;
    hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfEntry> g_prof;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t take_event() {
    if (!g_event_pool.empty()) {
        hipEvent_t e = g_event_pool.back();
        g_event_pool.pop_back();
        return e;
    }
    hipEvent_t e;
    GNNAV_HIP(hipEventCreate(&e));
    return e;
}

thread_local bool t_timers_off = false;
}  // namespace

namespace gnnav {
bool profiling_on() { return g_prof_on; }

KernelTimer::KernelTimer(const char *name, hipStream_t s) : stream(s) {
    if (!g_prof_on || t_timers_off) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    int idx = -1;
    for (size_t i = 0; i < g_prof.size(); ++i)
        if (g_prof[i].name == name) idx = (int)i;
    if (idx < 0) {
        g_prof.push_back(ProfEntry{name, 0, 0, {}});
        idx = (int)g_prof.size() - 1;
    }
    Pending p{idx, take_event(), take_event()};
    GNNAV_HIP(hipEventRecord(p.a, s));
    g_pending.push_back(p);
    slot = (int)g_pending.size() - 1;
}
KernelTimer::~KernelTimer() {
    if (slot < 0) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    (void)hipEventRecord(g_pending[slot].b, stream);
    g_prof[g_pending[slot].slot].launches++;
}
}  // namespace gnnav

// Turns per-kernel timing off on this thread while it lives.
struct TimersOff {
    bool prev;
    TimersOff() : prev(t_timers_off) { t_timers_off = true; }
    ~TimersOff() { t_timers_off = prev; }
};

// An empty kernel launched when recording starts (which = 1) and stops
// (which = 2): it marks the recorded region in an external kernel trace.
__global__ void k_profile_mark(int which) { (void)which; }

static void profile_mark(int which) {
    hipLaunchKernelGGL(k_profile_mark, dim3(1), dim3(64), 0, nullptr, which);
    GNNAV_HIP(hipGetLastError());
    GNNAV_HIP(hipDeviceSynchronize());
}

extern "C" gnnav_status gnnav_profile_start(void) {
    return guarded([&] {
        GNNAV_HIP(hipDeviceSynchronize());
        profile_mark(1);
        std::lock_guard<std::mutex> lk(g_prof_mu);
        for (auto &p : g_pending) {
            g_event_pool.push_back(p.a);
            g_event_pool.push_back(p.b);
        }
        g_pending.clear();
        g_prof.clear();
        g_prof_on = true;
    });
}

extern "C" gnnav_status gnnav_profile_stop(void) {
    return guarded([&] {
        GNNAV_HIP(hipDeviceSynchronize());
        profile_mark(2);
        std::lock_guard<std::mutex> lk(g_prof_mu);
        g_prof_on = false;
        for (auto &p : g_pending) {
            float ms = 0;
            GNNAV_HIP(hipEventElapsedTime(&ms, p.a, p.b));
            g_prof[p.slot].ms += ms;
            g_prof[p.slot].samples.push_back(ms);
            g_event_pool.push_back(p.a);
            g_event_pool.push_back(p.b);
        }
        g_pending.clear();
    });
}

extern "C" int32_t gnnav_profile_count(void) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    return (int32_t)g_prof.size();
}

extern "C" gnnav_status gnnav_profile_get(int32_t i, char *name, int32_t name_cap, int64_t *launches,
                                          double *total_ms) {
    return guarded([&] {
        std::lock_guard<std::mutex> lk(g_prof_mu);
        GNNAV_CHECK(i >= 0 && i < (int32_t)g_prof.size(), GNNAV_E_INVALID, "profile index out of range");
        if (name && name_cap > 0) {
            std::strncpy(name, g_prof[i].name.c_str(), (size_t)name_cap - 1);
            name[name_cap - 1] = 0;
        }
        if (launches) *launches = g_prof[i].launches;
        if (total_ms) *total_ms = g_prof[i].ms;
    });
}

extern "C" gnnav_status gnnav_profile_samples(int32_t i, float *ms, int64_t cap, int64_t *n) {
    return guarded([&] {
        std::lock_guard<std::mutex> lk(g_prof_mu);
        GNNAV_CHECK(i >= 0 && i < (int32_t)g_prof.size(), GNNAV_E_INVALID, "profile index out of range");
        GNNAV_CHECK(cap >= 0 && (cap == 0 || ms), GNNAV_E_INVALID, "NULL output with cap > 0");
        const auto &v = g_prof[i].samples;
        const int64_t k = std::min<int64_t>(cap, (int64_t)v.size());
        if (k > 0) std::memcpy(ms, v.data(), (size_t)k * sizeof(float));
        if (n) *n = (int64_t)v.size();
    });
}

// ------------------------------------------------------------------ graph
struct gnnav_graph {
    int64_t n = 0, nnz = 0, max_deg = 0;
    bool i64 = false;
    std::vector<int64_t> row_ptr_host;
    DevBuf row_ptr, col;
};

static void parallel_for(int64_t n, const std::function<void(int64_t, int64_t)> &fn) {
    unsigned hw = std::thread::hardware_concurrency();
    int64_t T = std::max<int64_t>(1, std::min<int64_t>(hw ? hw : 1, 16));
    if (n < 100000) T = 1;
    std::vector<std::thread> th;
    for (int64_t t = 0; t < T; ++t) {
        int64_t b = n * t / T, e = n * (t + 1) / T;
        if (t == T - 1)
            fn(b, e);
        else
            th.emplace_back(fn, b, e);
    }
    for (auto &x : th) x.join();
}

extern "C" gnnav_status gnnav_build_csr(int64_t n_nodes, int64_t n_edges, const int32_t *src,
                                        const int32_t *dst, uint32_t flags, gnnav_graph **out) {
    return guarded([&] {
        GNNAV_CHECK(out, GNNAV_E_INVALID, "out is NULL");
        GNNAV_CHECK(n_nodes >= 0 && n_nodes <= INT32_MAX, GNNAV_E_INVALID, "n_nodes outside [0, INT32_MAX]");
        GNNAV_CHECK(n_edges >= 0, GNNAV_E_INVALID, "n_edges < 0");
        GNNAV_CHECK(n_edges == 0 || (src && dst), GNNAV_E_INVALID, "src/dst NULL");
        const bool sym = flags & GNNAV_SYMMETRIZE;
        for (int64_t i = 0; i < n_edges; ++i)
            GNNAV_CHECK(src[i] >= 0 && src[i] < n_nodes && dst[i] >= 0 && dst[i] < n_nodes, GNNAV_E_RANGE,
                        "edge " + std::to_string(i) + " has an endpoint outside [0, n_nodes)");
        // bucket the arcs by source row (counting sort), then sort + dedup each row
        std::vector<int64_t> rp(n_nodes + 1, 0);
        for (int64_t i = 0; i < n_edges; ++i) {
            if (src[i] == dst[i]) continue;
            rp[src[i] + 1]++;
            if (sym) rp[dst[i] + 1]++;
        }
        for (int64_t v = 0; v < n_nodes; ++v) rp[v + 1] += rp[v];
        std::vector<int32_t> col(std::max<int64_t>(rp[n_nodes], 1));
        {
            std::vector<int64_t> fill(rp.begin(), rp.end() - 1);
            for (int64_t i = 0; i < n_edges; ++i) {
                if (src[i] == dst[i]) continue;
                col[fill[src[i]]++] = dst[i];
                if (sym) col[fill[dst[i]]++] = src[i];
            }
        }
        std::vector<int64_t> kept(n_nodes + 1, 0);
        parallel_for(n_nodes, [&](int64_t b, int64_t e) {
            for (int64_t v = b; v < e; ++v) {
                int32_t *r0 = col.data() + rp[v], *r1 = col.data() + rp[v + 1];
                std::sort(r0, r1);
                kept[v + 1] = std::unique(r0, r1) - r0;
            }
        });
        auto *g = new gnnav_graph();
        try {
            g->n = n_nodes;
            g->row_ptr_host.assign(n_nodes + 1, 0);
            for (int64_t v = 0; v < n_nodes; ++v) {
                g->row_ptr_host[v + 1] = g->row_ptr_host[v] + kept[v + 1];
                g->max_deg = std::max<int64_t>(g->max_deg, kept[v + 1]);
            }
            g->nnz = g->row_ptr_host[n_nodes];
            for (int64_t v = 0, o = 0; v < n_nodes; ++v) {  // compact rows in place (o <= rp[v])
                std::memmove(col.data() + o, col.data() + rp[v], (size_t)kept[v + 1] * sizeof(int32_t));
                o += kept[v + 1];
            }
            g->i64 = (flags & GNNAV_OFFSETS_I64) || g->nnz > INT32_MAX;
            hipStream_t s0 = nullptr;
            if (g->i64) {
                g->row_ptr.ensure((n_nodes + 1) * sizeof(int64_t), s0);
                GNNAV_HIP(hipMemcpy(g->row_ptr.p, g->row_ptr_host.data(), (n_nodes + 1) * sizeof(int64_t),
                                    hipMemcpyHostToDevice));
            } else {
                std::vector<int32_t> r32(g->row_ptr_host.begin(), g->row_ptr_host.end());
                g->row_ptr.ensure((n_nodes + 1) * sizeof(int32_t), s0);
                GNNAV_HIP(hipMemcpy(g->row_ptr.p, r32.data(), (n_nodes + 1) * sizeof(int32_t),
                                    hipMemcpyHostToDevice));
            }
            g->col.ensure(std::max<int64_t>(g->nnz, 1) * sizeof(int32_t), s0);
            if (g->nnz > 0)
                GNNAV_HIP(hipMemcpy(g->col.p, col.data(), g->nnz * sizeof(int32_t), hipMemcpyHostToDevice));
        } catch (...) {
            g->row_ptr.release();
            g->col.release();
            delete g;
            throw;
        }
        *out = g;
    });
}

extern "C" gnnav_status gnnav_graph_info(const gnnav_graph *g, int64_t *n_nodes, int64_t *nnz,
                                         int64_t *max_degree, int32_t *offsets_i64) {
    return guarded([&] {
        GNNAV_CHECK(g, GNNAV_E_INVALID, "graph is NULL");
        if (n_nodes) *n_nodes = g->n;
        if (nnz) *nnz = g->nnz;
        if (max_degree) *max_degree = g->max_deg;
        if (offsets_i64) *offsets_i64 = g->i64 ? 1 : 0;
    });
}

extern "C" gnnav_status gnnav_graph_csr_host(const gnnav_graph *g, int64_t *row_ptr, int32_t *col) {
    return guarded([&] {
        GNNAV_CHECK(g && row_ptr, GNNAV_E_INVALID, "NULL argument");
        std::memcpy(row_ptr, g->row_ptr_host.data(), (g->n + 1) * sizeof(int64_t));
        if (col && g->nnz > 0) GNNAV_HIP(hipMemcpy(col, g->col.p, g->nnz * sizeof(int32_t), hipMemcpyDeviceToHost));
    });
}

extern "C" void gnnav_graph_free(gnnav_graph *g) {
    if (!g) return;
    (void)hipDeviceSynchronize();
    g->row_ptr.release();
    g->col.release();
    delete g;
}

static bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// ------------------------------------------------------------------ cache
constexpr int64_t kStoreAlign = 128;  // host store row alignment, bytes (one L2 line)
// Scratch of one gather in flight: hit/miss lists, scan partials, device
// counts, and the second stream that carries the miss copy.  Each caller
// stream gets its own, so gathers on different streams may overlap.
struct GatherWs {
    hipStream_t stream = nullptr;
    DevBuf hit_list, miss_list, dev_counts;
    ScanState scan;
};

struct gnnav_cache {
    int64_t n = 0, c = 0, d = 0, ld = 0, elt = 4;
    gnnav_dtype dt = GNNAV_F32;
    bool store_on_device = false;
    DevBuf slot_map, cache_rows, store_dev;
    void *store_host = nullptr;       // pinned, device-mapped
    void *store_ptr = nullptr;        // device-visible address of the store
    int64_t store_pitch = 0;          // store row stride in bytes
    std::vector<int32_t> slot_host;
    std::vector<int32_t> rank_host;   // degree rank (first C fill the cache)
    std::mutex ws_mu;
    std::vector<GatherWs *> ws;
    int32_t link_wgs = 64;            // workgroups copying misses over the host link
    // update policy (GNNAV_POLICY_*) over the ring of slots [ring_lo, c):
    // FIFO's ring pointer, LRU's recency list, stamps and partition scan
    int32_t policy = 0;
    int64_t ring_lo = 0, ring_n = 0;
    DevBuf owner, ring_ptr;   // FIFO: two pointer words, ring_parity the current one
    bool owner_filled = false;   // owner holds the degree ranking (or later contents)
    int ring_parity = 0;
    DevBuf lru_order, lru_part, lru_stamp, lru_ctl;
    ScanState lru_scan;
    std::mutex upd_mu;
    hipEvent_t upd_done = nullptr;
    bool upd_recorded = false;
    // adjacency partitioned by this cache's (static) slot map, for the
    // biased sampler; built on first use for a graph
    DevBuf part_col, part_cnt;
    const void *part_graph = nullptr;
    int64_t part_nnz = -1;
    hipEvent_t part_ready = nullptr;
};

static GatherWs *gather_ws(gnnav_cache *c, hipStream_t s) {
    std::lock_guard<std::mutex> lk(c->ws_mu);
    for (auto *w : c->ws)
        if (w->stream == s) return w;
    auto *w = new GatherWs();
    w->stream = s;
    c->ws.push_back(w);
    return w;
}

static void free_cache(gnnav_cache *c) {
    if (!c) return;
    (void)hipDeviceSynchronize();
    c->slot_map.release();
    c->cache_rows.release();
    c->store_dev.release();
    for (auto *w : c->ws) {
        w->hit_list.release();
        w->miss_list.release();
        w->dev_counts.release();
        w->scan.release();
        delete w;
    }
    c->owner.release();
    c->ring_ptr.release();
    c->lru_order.release();
    c->lru_part.release();
    c->lru_stamp.release();
    c->lru_ctl.release();
    c->lru_scan.release();
    c->part_col.release();
    c->part_cnt.release();
    if (c->part_ready) (void)hipEventDestroy(c->part_ready);
    if (c->upd_done) (void)hipEventDestroy(c->upd_done);
    if (c->store_host) (void)hipHostFree(c->store_host);
    delete c;
}

// Copy rows ids[0..count) (or rows 0..count) of the padded host image into
// device memory through a pinned staging buffer.
static void upload_rows(void *dst_dev, const uint8_t *feats, int64_t row_bytes, int64_t pitch,
                        const int32_t *ids, int64_t count) {
    if (count <= 0) return;
    const int64_t chunk_rows = std::max<int64_t>(1, (64 << 20) / pitch);
    void *stage = nullptr;
    host_pinned_alloc(&stage, (size_t)(chunk_rows * pitch), hipHostMallocDefault, "upload staging");
    try {
        for (int64_t r0 = 0; r0 < count; r0 += chunk_rows) {
            const int64_t rn = std::min(chunk_rows, count - r0);
            uint8_t *sp = (uint8_t *)stage;
            std::memset(sp, 0, (size_t)(rn * pitch));
            for (int64_t i = 0; i < rn; ++i) {
                const int64_t v = ids ? ids[r0 + i] : r0 + i;
                std::memcpy(sp + i * pitch, feats + v * row_bytes, (size_t)row_bytes);
            }
            GNNAV_HIP(hipMemcpy((uint8_t *)dst_dev + r0 * pitch, stage, (size_t)(rn * pitch),
                                hipMemcpyHostToDevice));
        }
    } catch (...) {
        (void)hipHostFree(stage);
        throw;
    }
    GNNAV_HIP(hipHostFree(stage));
}

extern "C" gnnav_status gnnav_build_cache(const gnnav_graph *g, const void *feats_host, int64_t d, gnnav_dtype dt,
                                          double cache_fraction, uint32_t flags, gnnav_cache **out) {
    return guarded([&] {
        GNNAV_CHECK(g && out, GNNAV_E_INVALID, "NULL graph or out");
        GNNAV_CHECK(d > 0, GNNAV_E_INVALID, "d must be positive");
        GNNAV_CHECK(dt == GNNAV_F32 || dt == GNNAV_BF16, GNNAV_E_INVALID, "dtype must be F32 or BF16");
        GNNAV_CHECK(cache_fraction >= 0.0 && cache_fraction <= 1.0, GNNAV_E_INVALID,
                    "cache_fraction outside [0, 1]");
        GNNAV_CHECK(g->n == 0 || feats_host, GNNAV_E_INVALID, "feats_host is NULL");
        auto *c = new gnnav_cache();
        try {
            c->n = g->n;
            c->d = d;
            c->dt = dt;
            c->elt = dt == GNNAV_BF16 ? 2 : 4;
            const int64_t row_bytes = d * c->elt;
            const int64_t pitch = (row_bytes + 15) / 16 * 16;
            c->ld = pitch / c->elt;
            c->store_on_device = flags & GNNAV_STORE_ON_DEVICE;
            // degree ranking: degree descending, id ascending (counting sort)
            const int64_t n = g->n;
            std::vector<int64_t> bucket(g->max_deg + 2, 0);
            for (int64_t v = 0; v < n; ++v) bucket[g->max_deg - (g->row_ptr_host[v + 1] - g->row_ptr_host[v]) + 1]++;
            for (size_t i = 1; i < bucket.size(); ++i) bucket[i] += bucket[i - 1];
            std::vector<int32_t> rank(std::max<int64_t>(n, 1));
            for (int64_t v = 0; v < n; ++v)
                rank[bucket[g->max_deg - (g->row_ptr_host[v + 1] - g->row_ptr_host[v])]++] = (int32_t)v;
            int64_t C = (int64_t)std::floor(cache_fraction * (double)n);
            C = std::max<int64_t>(0, std::min<int64_t>(C, n));
            c->c = C;
            c->slot_host.assign(n, -1);
            for (int64_t s = 0; s < C; ++s) c->slot_host[rank[s]] = (int32_t)s;
            c->rank_host.assign(rank.begin(), rank.begin() + C);
            hipStream_t s0 = nullptr;
            c->slot_map.ensure(std::max<int64_t>(n, 1) * sizeof(int32_t), s0);
            if (n > 0)
                GNNAV_HIP(hipMemcpy(c->slot_map.p, c->slot_host.data(), n * sizeof(int32_t), hipMemcpyHostToDevice));
            const uint8_t *feats = (const uint8_t *)feats_host;
            c->cache_rows.ensure(std::max<int64_t>(C, 1) * pitch, s0);
            upload_rows(c->cache_rows.p, feats, row_bytes, pitch, rank.data(), C);
            if (c->store_on_device) {
                c->store_pitch = pitch;
                c->store_dev.ensure(std::max<int64_t>(n, 1) * pitch, s0);
                upload_rows(c->store_dev.p, feats, row_bytes, pitch, nullptr, n);
                c->store_ptr = c->store_dev.p;
            } else {
                // Rows of the host store start on kStoreAlign-byte boundaries:
                // the zero-copy reads of a miss then cross as few of the
                // link's read blocks as the row's length allows.
                const int64_t sp = (row_bytes + kStoreAlign - 1) / kStoreAlign * kStoreAlign;
                c->store_pitch = sp;
                const size_t bytes = (size_t)std::max<int64_t>(n, 1) * sp;
                host_pinned_alloc(&c->store_host, bytes, hipHostMallocMapped, "feature store");
                uint8_t *hp = (uint8_t *)c->store_host;
                parallel_for(n, [&](int64_t b, int64_t e) {
                    for (int64_t v = b; v < e; ++v) {
                        std::memcpy(hp + v * sp, feats + v * row_bytes, (size_t)row_bytes);
                        std::memset(hp + v * sp + row_bytes, 0, (size_t)(sp - row_bytes));
                    }
                });
                GNNAV_HIP(hipHostGetDevicePointer(&c->store_ptr, c->store_host, 0));
            }
        } catch (...) {
            free_cache(c);
            throw;
        }
        *out = c;
    });
}

extern "C" gnnav_status gnnav_cache_info(const gnnav_cache *c, int64_t *n_cached, int64_t *d, int64_t *ld,
                                         int32_t *dtype, int32_t *store_on_device) {
    return guarded([&] {
        GNNAV_CHECK(c, GNNAV_E_INVALID, "cache is NULL");
        if (n_cached) *n_cached = c->c;
        if (d) *d = c->d;
        if (ld) *ld = c->ld;
        if (dtype) *dtype = (int32_t)c->dt;
        if (store_on_device) *store_on_device = c->store_on_device ? 1 : 0;
    });
}

extern "C" gnnav_status gnnav_cache_slot_map_host(const gnnav_cache *c, int32_t *slot_map) {
    return guarded([&] {
        GNNAV_CHECK(c && slot_map, GNNAV_E_INVALID, "NULL argument");
        GNNAV_HIP(hipDeviceSynchronize());
        if (c->n > 0)
            GNNAV_HIP(hipMemcpy(slot_map, c->slot_map.p, c->n * sizeof(int32_t), hipMemcpyDeviceToHost));
    });
}

extern "C" gnnav_status gnnav_cache_contents_host(const gnnav_cache *c, int32_t *owners, void *rows) {
    return guarded([&] {
        GNNAV_CHECK(c, GNNAV_E_INVALID, "cache is NULL");
        GNNAV_HIP(hipDeviceSynchronize());
        if (owners) {
            if (c->owner_filled) {
                if (c->c > 0)
                    GNNAV_HIP(hipMemcpy(owners, c->owner.p, c->c * sizeof(int32_t), hipMemcpyDeviceToHost));
            } else {
                std::memcpy(owners, c->rank_host.data(), c->c * sizeof(int32_t));
            }
        }
        if (rows && c->c > 0)
            GNNAV_HIP(hipMemcpy(rows, c->cache_rows.p, (size_t)(c->c * c->ld * c->elt), hipMemcpyDeviceToHost));
    });
}

extern "C" gnnav_status gnnav_cache_set_link_workgroups(gnnav_cache *c, int32_t workgroups) {
    return guarded([&] {
        GNNAV_CHECK(c, GNNAV_E_INVALID, "cache is NULL");
        GNNAV_CHECK(workgroups >= 1 && workgroups <= 4096, GNNAV_E_INVALID, "workgroups outside [1, 4096]");
        c->link_wgs = workgroups;
    });
}

extern "C" gnnav_status gnnav_cache_set_policy(gnnav_cache *c, int32_t policy, int64_t dynamic_slots) {
    return guarded([&] {
        GNNAV_CHECK(c, GNNAV_E_INVALID, "cache is NULL");
        GNNAV_CHECK(policy == GNNAV_POLICY_STATIC || policy == GNNAV_POLICY_FIFO || policy == GNNAV_POLICY_LRU,
                    GNNAV_E_INVALID, "unknown policy");
        GNNAV_CHECK(policy == GNNAV_POLICY_STATIC || (dynamic_slots >= 0 && dynamic_slots <= c->c), GNNAV_E_INVALID,
                    "dynamic_slots outside [0, cached rows]");
        GNNAV_HIP(hipDeviceSynchronize());
        std::lock_guard<std::mutex> lk(c->upd_mu);
        const int64_t rn = policy == GNNAV_POLICY_STATIC ? 0 : dynamic_slots, lo = c->c - rn;
        // The cache reads as static until the ring's state is in place, so a
        // call that fails here (E_NOMEM) leaves it static, never pointing a
        // gather at buffers that are missing or not yet filled.
        c->policy = GNNAV_POLICY_STATIC;
        c->ring_n = 0;
        c->ring_lo = c->c;
        c->part_graph = nullptr;   // the slot map may have moved: rebuild the partition on next use
        if (rn > 0) {
            hipStream_t s0 = nullptr;
            if (!c->owner_filled) {
                // first dynamic use: owner table from the degree ranking
                c->owner.ensure(std::max<int64_t>(c->c, 1) * sizeof(int32_t), s0);
                GNNAV_HIP(hipMemcpy(c->owner.p, c->rank_host.data(), c->c * sizeof(int32_t), hipMemcpyHostToDevice));
                c->owner_filled = true;
            }
            c->ring_ptr.ensure(2 * sizeof(int32_t), s0);
            GNNAV_HIP(hipMemset(c->ring_ptr.p, 0, 2 * sizeof(int32_t)));
            c->ring_parity = 0;
            if (policy == GNNAV_POLICY_LRU) {
                // recency starts in slot order (lowest ring slot least
                // recent); `part` starts as a copy, so it only ever holds ring
                // slots, even where a partition scan that gave up left a gap
                const size_t bytes = (size_t)rn * sizeof(int32_t);
                c->lru_order.ensure(bytes, s0);
                c->lru_part.ensure(bytes, s0);
                c->lru_stamp.ensure(bytes, s0);
                c->lru_ctl.ensure(3 * sizeof(uint32_t), s0);
                std::vector<int32_t> order((size_t)rn);
                for (int64_t j = 0; j < rn; ++j) order[(size_t)j] = (int32_t)(lo + j);
                GNNAV_HIP(hipMemcpy(c->lru_order.p, order.data(), bytes, hipMemcpyHostToDevice));
                GNNAV_HIP(hipMemcpy(c->lru_part.p, order.data(), bytes, hipMemcpyHostToDevice));
                GNNAV_HIP(hipMemset(c->lru_stamp.p, 0, bytes));
                GNNAV_HIP(hipMemset(c->lru_ctl.p, 0, 3 * sizeof(uint32_t)));
                c->lru_scan.ensure(rn, s0);
            }
            GNNAV_HIP(hipDeviceSynchronize());
            if (!c->upd_done) GNNAV_HIP(hipEventCreateWithFlags(&c->upd_done, hipEventDisableTiming));
            c->upd_recorded = false;
        }
        c->policy = policy;
        c->ring_n = rn;
        c->ring_lo = lo;
    });
}

extern "C" void gnnav_cache_free(gnnav_cache *c) { free_cache(c); }

// ----------------------------------------------------------------- blocks
namespace {
constexpr int kMaxHops = 16;
constexpr int32_t kSlotFanout = 64;   // largest fanout sampled into slot lists
constexpr int kSizeN = 0;         // sizes[kSizeN + h] = |F_h|
constexpr int kSizeE = 17;        // sizes[kSizeE + h] = E_h (h >= 1)
constexpr int kSizeErr = 40;      // out-of-range seed count: slot 40 + (call parity)
constexpr int kSizeSlots = 48;
}  // namespace

struct gnnav_blocks {
    int32_t L = 0;
    bool host_sizes = false;           // n_h / e_h hold the last sample's sizes
    int64_t n_h[kMaxHops + 1] = {0};
    int64_t e_h[kMaxHops + 1] = {0};
    int64_t nb[kMaxHops + 1] = {0};    // Eq. 12 capacity bounds of the last sample
    int64_t eb[kMaxHops + 1] = {0};
    int64_t map_nodes = -1;
    uint64_t calls = 0;                // sampling calls; their parity picks the error-count slot
    uint32_t map_epoch = 0;            // sampling calls since the node table was last filled
    DevBuf map, sizes, nodes;
    ScanState scan;
    DevBuf indptr[kMaxHops], nbrs[kMaxHops], indices[kMaxHops];
    DevBuf slots[kMaxHops];            // slot lists of hops with 0 < k <= 64
    int32_t *sizes_host = nullptr;  // pinned mirror of `sizes`
    DevBuf agg, hid[2];             // forward workspace
    // training: activations kept per layer, gradients, transposed blocks
    DevBuf act_agg[kMaxHops], act_h[kMaxHops];
    DevBuf dz[2], dself, dagg, wpart, row_loss, dw_tmp;
    CscWorkspace csc;
};

extern "C" gnnav_status gnnav_blocks_create(gnnav_blocks **out) {
    return guarded([&] {
        GNNAV_CHECK(out, GNNAV_E_INVALID, "out is NULL");
        auto *b = new gnnav_blocks();
        try {
            host_pinned_alloc((void **)&b->sizes_host, (kSizeSlots + 1) * sizeof(int32_t), hipHostMallocDefault,
                              "size mirror");
        } catch (...) {
            delete b;
            throw;
        }
        *out = b;
    });
}

extern "C" void gnnav_blocks_free(gnnav_blocks *b) {
    if (!b) return;
    (void)hipDeviceSynchronize();
    b->map.release();
    b->sizes.release();
    b->nodes.release();
    b->scan.release();
    for (int h = 0; h < kMaxHops; ++h) {
        b->indptr[h].release();
        b->nbrs[h].release();
        b->indices[h].release();
        b->slots[h].release();
    }
    b->agg.release();
    b->hid[0].release();
    b->hid[1].release();
    for (int h = 0; h < kMaxHops; ++h) {
        b->act_agg[h].release();
        b->act_h[h].release();
    }
    for (DevBuf *d : {&b->dz[0], &b->dz[1], &b->dself, &b->dagg, &b->wpart, &b->row_loss, &b->dw_tmp}) d->release();
    b->csc.release();
    if (b->sizes_host) (void)hipHostFree(b->sizes_host);
    delete b;
}

// Enqueues the whole expansion on `s`; sizes stay in device memory.
static void sample_enqueue(const gnnav_graph *g, const int32_t *seeds_dev, int64_t n_seeds, const int32_t *fanouts,
                           int32_t n_hops, uint64_t rng_seed, gnnav_blocks *b, hipStream_t s,
                           const gnnav_cache *bias = nullptr, uint32_t eta = 1) {
    // Every argument and capacity check comes before any state changes, so a
    // call that fails here leaves the blocks (and the cache) as they were.
    GNNAV_CHECK(g && b && fanouts, GNNAV_E_INVALID, "NULL graph, blocks or fanouts");
    GNNAV_CHECK(n_hops >= 1 && n_hops <= kMaxHops, GNNAV_E_INVALID, "n_hops outside [1, 16]");
    GNNAV_CHECK(n_seeds >= 0, GNNAV_E_INVALID, "n_seeds < 0");
    GNNAV_CHECK(n_seeds == 0 || seeds_dev, GNNAV_E_INVALID, "seeds_dev is NULL");
    GNNAV_CHECK(n_seeds <= INT32_MAX, GNNAV_E_CAPACITY, "n_seeds above INT32_MAX");
    for (int h = 0; h < n_hops; ++h)
        GNNAV_CHECK(fanouts[h] <= 1024, GNNAV_E_INVALID, "fanout above 1024");
    if (bias) {
        GNNAV_CHECK(bias->n == g->n, GNNAV_E_INVALID, "the cache belongs to a graph of another size");
        GNNAV_CHECK(eta >= 1 && eta <= 65536, GNNAV_E_INVALID, "eta outside [1, 65536]");
        for (int h = 0; h < n_hops; ++h)
            GNNAV_CHECK(fanouts[h] <= 64, GNNAV_E_INVALID, "biased sampling supports fanouts up to 64");
    }
    // Eq. 12 capacity bounds (tau = 1, no overlap): E_h <= n_(h-1) * k_h,
    // n_h <= min(n, n_(h-1) + E_h).
    int64_t nb[kMaxHops + 1], eb[kMaxHops + 1];
    // Hops with 0 < k <= 64 sample into slot lists of stride min(k, max
    // degree) (no count scan before them); the stride is also their per-row
    // edge bound.
    int32_t stride[kMaxHops + 1] = {0};
    nb[0] = std::min<int64_t>(n_seeds, g->n);
    eb[0] = 0;
    for (int h = 1; h <= n_hops; ++h) {
        const int64_t k = fanouts[h - 1] < 0 ? g->max_deg : std::min<int64_t>(fanouts[h - 1], g->max_deg);
        if (fanouts[h - 1] > 0 && fanouts[h - 1] <= kSlotFanout && k > 0) stride[h] = (int32_t)k;
        eb[h] = nb[h - 1] * k;
        nb[h] = std::min<int64_t>(g->n, nb[h - 1] + eb[h]);
        GNNAV_CHECK(eb[h] < INT32_MAX && nb[h] < INT32_MAX, GNNAV_E_CAPACITY,
                    "hop " + std::to_string(h) + " bound exceeds the int32 range");
    }
    if (bias) {
        auto *bc = const_cast<gnnav_cache *>(bias);
        std::lock_guard<std::mutex> lk(bc->upd_mu);
        if (bc->ring_n > 0) {
            // a self-updating cache: read its slot map after the last update
            if (bc->upd_recorded) GNNAV_HIP(hipStreamWaitEvent(s, bc->upd_done, 0));
        } else {
            // a static cache: rows partitioned by its slot map, built once per graph
            if (bc->part_graph != (const void *)g || bc->part_nnz != g->nnz) {
                bc->part_graph = nullptr;   // a failed reallocation below has freed the old partition
                bc->part_col.ensure(std::max<int64_t>(g->nnz, 1) * sizeof(int32_t), s);
                bc->part_cnt.ensure(std::max<int64_t>(g->n, 1) * sizeof(int32_t), s);
                launch_partition_rows(g->row_ptr.p, g->i64, g->col.as<int32_t>(), g->n, bc->slot_map.as<int32_t>(),
                                      bc->part_col.as<int32_t>(), bc->part_cnt.as<int32_t>(), s);
                if (!bc->part_ready) GNNAV_HIP(hipEventCreateWithFlags(&bc->part_ready, hipEventDisableTiming));
                GNNAV_HIP(hipEventRecord(bc->part_ready, s));
                bc->part_graph = g;
                bc->part_nnz = g->nnz;
            } else {
                GNNAV_HIP(hipStreamWaitEvent(s, bc->part_ready, 0));
            }
        }
    }
    int64_t max_list = n_seeds;
    for (int h = 1; h <= n_hops; ++h) max_list = std::max(max_list, std::max(eb[h], nb[h - 1] + 1));
    // workspace: growing it frees the previous sample's buffers, so until
    // this sample is enqueued the blocks read as unsampled (a call that fails
    // below, E_NOMEM, leaves nothing that points at freed memory)
    b->L = 0;
    b->host_sizes = false;
    // node table: all-ones entries are older than every call's tag; after
    // 2^32 - 2 calls the tags would wrap, so the table is filled again
    if (b->map_nodes < g->n || b->map_epoch == 0xfffffffeu) {
        b->map_nodes = 0;   // a failed reallocation below has freed the old table
        b->map.ensure(std::max<int64_t>(g->n, 1) * sizeof(uint64_t), s);
        launch_fill_i32(b->map.as<int32_t>(), -1, 2 * std::max<int64_t>(g->n, 1), s);
        b->map_nodes = g->n;
        b->map_epoch = 0;
    }
    const uint32_t tag = 0xffffffffu - ++b->map_epoch;
    if (!b->sizes.p) {
        b->sizes.ensure(kSizeSlots * sizeof(int32_t), s);
        launch_fill_i32(b->sizes.as<int32_t>(), 0, kSizeSlots, s);   // once: both error-count slots start at 0
    }
    b->nodes.ensure(std::max<int64_t>(nb[n_hops], 1) * sizeof(int32_t), s);
    b->scan.ensure(max_list, s);
    for (int h = 1; h <= n_hops; ++h) {
        b->indptr[h - 1].ensure((nb[h - 1] + 1) * sizeof(int32_t), s);
        b->nbrs[h - 1].ensure(std::max<int64_t>(eb[h], 1) * sizeof(int32_t), s);
        b->indices[h - 1].ensure(std::max<int64_t>(eb[h], 1) * sizeof(int32_t), s);
        if (stride[h]) b->slots[h - 1].ensure(std::max<int64_t>(eb[h], 1) * sizeof(int32_t), s);
    }
    int32_t *sz = b->sizes.as<int32_t>();
    uint64_t *map = b->map.as<uint64_t>();
    int32_t *nodes = b->nodes.as<int32_t>();
    // Every size slot is written by this call's scans; the out-of-range seed
    // count alternates between two slots, the other one cleared by this call
    // for the next (so no clearing launch is needed).
    const int par = (int)(++b->calls & 1);
    // F_0 (seeds without repeats, first occurrence kept), with hop 1's row
    // counts (indptr_1, E_1) in the same scan unless hop 1 uses a slot list
    DedupArgs d0{seeds_dev, n_seeds, nullptr, n_seeds, map, tag, g->n, nodes, nullptr, sz + kSizeN,
                 sz + kSizeErr + par, &b->scan};
    d0.err_next = sz + kSizeErr + (par ^ 1);
    if (!stride[1]) {
        d0.count_row_ptr = g->row_ptr.p;
        d0.count_i64 = g->i64;
        d0.count_k = fanouts[0];
        d0.count_indptr = b->indptr[0].as<int32_t>();
        d0.count_e_out = sz + kSizeE + 1;
    }
    launch_dedup(d0, s);
    for (int h = 1; h <= n_hops; ++h) {
        const bool slotted = stride[h] > 0;
        SampleHopArgs a{g->row_ptr.p, g->i64, g->col.as<int32_t>(), nodes, sz + kSizeN + h - 1,
                        b->indptr[h - 1].as<int32_t>(), (slotted ? b->slots : b->nbrs)[h - 1].as<int32_t>(),
                        sz + kSizeE + h, fanouts[h - 1], rng_seed, (uint32_t)(h - 1), nb[h - 1], &b->scan,
                        bias ? bias->slot_map.as<int32_t>() : nullptr, eta,
                        bias && bias->ring_n == 0 ? bias->part_col.as<int32_t>() : nullptr,
                        bias && bias->ring_n == 0 ? bias->part_cnt.as<int32_t>() : nullptr, map, tag};
        a.slot_stride = stride[h];
        a.n_nodes = g->n;
        // hop h - 1's relabel rides along with this hop's first scan
        const int32_t *rl_list = h > 1 ? b->nbrs[h - 2].as<int32_t>() : nullptr;
        if (!slotted) {
            if (rl_list) {
                a.relabel_list = rl_list;
                a.relabel_len = sz + kSizeE + h - 1;
                a.relabel_bound = eb[h - 1];
                a.relabel_n = sz + kSizeN + h - 1;
                a.relabel_indices = b->indices[h - 2].as<int32_t>();
            }
            if (h > 1) launch_count_scan(a, s);   // hop 1's ran with the seeds' dedup
        }
        launch_sample_hop(a, s);
        DedupArgs dh{(slotted ? b->slots : b->nbrs)[h - 1].as<int32_t>(), 0, sz + kSizeE + h, eb[h], map, tag,
                     g->n, nodes, sz + kSizeN + h - 1, sz + kSizeN + h, nullptr, &b->scan, true};
        if (slotted) {
            dh.len_ptr = nullptr;
            dh.slot_stride = stride[h];
            dh.compact_out = b->nbrs[h - 1].as<int32_t>();
            dh.indptr_out = b->indptr[h - 1].as<int32_t>();
            dh.e_out = sz + kSizeE + h;
            if (rl_list) {
                dh.relabel_list = rl_list;
                dh.relabel_len = sz + kSizeE + h - 1;
                dh.relabel_bound = eb[h - 1];
                dh.relabel_n = sz + kSizeN + h - 1;
                dh.relabel_indices = b->indices[h - 2].as<int32_t>();
            }
        }
        launch_dedup(dh, s);
    }
    launch_relabel(b->nbrs[n_hops - 1].as<int32_t>(), sz + kSizeE + n_hops, eb[n_hops], map, g->n,
                   sz + kSizeN + n_hops, b->indices[n_hops - 1].as<int32_t>(), s);
    b->L = n_hops;
    b->host_sizes = false;
    for (int h = 0; h <= n_hops; ++h) {
        b->nb[h] = nb[h];
        b->eb[h] = eb[h];
    }
}

// Copies the device sizes of the last sample to the host (waits on `s`).
static void publish_sizes(gnnav_blocks *b, hipStream_t s) {
    GNNAV_CHECK(b->sizes.p, GNNAV_E_INVALID, "blocks have not been sampled");
    GNNAV_HIP(hipMemcpyAsync(b->sizes_host, b->sizes.p, kSizeSlots * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    check_device_errors(s);   // also waits for s
    for (int h = 0; h <= b->L; ++h) b->n_h[h] = b->sizes_host[kSizeN + h];
    for (int h = 1; h <= b->L; ++h) b->e_h[h] = b->sizes_host[kSizeE + h];
    b->host_sizes = true;
    const int32_t bad = b->sizes_host[kSizeErr + (int)(b->calls & 1)];
    GNNAV_CHECK(bad == 0, GNNAV_E_RANGE, std::to_string(bad) + " seed(s) outside [0, n)");
}

extern "C" gnnav_status gnnav_sample(const gnnav_graph *g, const int32_t *seeds_dev, int64_t n_seeds,
                                     const int32_t *fanouts, int32_t n_hops, uint64_t rng_seed,
                                     gnnav_blocks *b, void *stream) {
    return guarded([&] {
        sample_enqueue(g, seeds_dev, n_seeds, fanouts, n_hops, rng_seed, b, (hipStream_t)stream);
        publish_sizes(b, (hipStream_t)stream);
    });
}

extern "C" gnnav_status gnnav_sample_async(const gnnav_graph *g, const int32_t *seeds_dev, int64_t n_seeds,
                                           const int32_t *fanouts, int32_t n_hops, uint64_t rng_seed,
                                           gnnav_blocks *b, void *stream) {
    return guarded([&] { sample_enqueue(g, seeds_dev, n_seeds, fanouts, n_hops, rng_seed, b, (hipStream_t)stream); });
}

extern "C" gnnav_status gnnav_sample_biased(const gnnav_graph *g, const gnnav_cache *cache, uint32_t eta,
                                            const int32_t *seeds_dev, int64_t n_seeds, const int32_t *fanouts,
                                            int32_t n_hops, uint64_t rng_seed, gnnav_blocks *b, int32_t async,
                                            void *stream) {
    return guarded([&] {
        GNNAV_CHECK(cache, GNNAV_E_INVALID, "cache is NULL");
        sample_enqueue(g, seeds_dev, n_seeds, fanouts, n_hops, rng_seed, b, (hipStream_t)stream, cache, eta);
        if (!async) publish_sizes(b, (hipStream_t)stream);
    });
}

extern "C" gnnav_status gnnav_blocks_sync(gnnav_blocks *b, void *stream) {
    return guarded([&] {
        GNNAV_CHECK(b, GNNAV_E_INVALID, "blocks is NULL");
        publish_sizes(b, (hipStream_t)stream);
    });
}

extern "C" gnnav_status gnnav_blocks_device_sizes(const gnnav_blocks *b, const int32_t **sizes_dev,
                                                  int64_t *bounds) {
    return guarded([&] {
        GNNAV_CHECK(b && sizes_dev, GNNAV_E_INVALID, "NULL argument");
        GNNAV_CHECK(b->sizes.p, GNNAV_E_INVALID, "blocks have not been sampled");
        *sizes_dev = b->sizes.as<int32_t>();
        if (bounds)
            for (int h = 0; h <= b->L; ++h) bounds[h] = b->nb[h];
    });
}

extern "C" gnnav_status gnnav_blocks_hop(const gnnav_blocks *b, int32_t hop, gnnav_block_view *out) {
    return guarded([&] {
        GNNAV_CHECK(b && out, GNNAV_E_INVALID, "NULL argument");
        GNNAV_CHECK(hop >= 1 && hop <= b->L, GNNAV_E_INVALID, "hop outside [1, L]");
        GNNAV_CHECK(b->host_sizes, GNNAV_E_INVALID, "sizes not on the host yet: call gnnav_blocks_sync");
        out->n_dst = b->n_h[hop - 1];
        out->n_src = b->n_h[hop];
        out->nnz = b->e_h[hop];
        out->indptr = b->indptr[hop - 1].as<int32_t>();
        out->indices = b->indices[hop - 1].as<int32_t>();
        out->neighbors = b->nbrs[hop - 1].as<int32_t>();
        out->src_ids = b->nodes.as<int32_t>();
    });
}

extern "C" gnnav_status gnnav_blocks_nodes(const gnnav_blocks *b, const int32_t **nodes_dev, int64_t *n_per_hop,
                                           int32_t *n_hops) {
    return guarded([&] {
        GNNAV_CHECK(b, GNNAV_E_INVALID, "blocks is NULL");
        GNNAV_CHECK(!n_per_hop || b->host_sizes, GNNAV_E_INVALID,
                    "sizes not on the host yet: call gnnav_blocks_sync");
        if (nodes_dev) *nodes_dev = b->nodes.as<int32_t>();
        if (n_per_hop)
            for (int h = 0; h <= b->L; ++h) n_per_hop[h] = b->n_h[h];
        if (n_hops) *n_hops = b->L;
    });
}

// ----------------------------------------------------------------- gather

// `fixed`: a workspace to use instead of the stream's own (the no-allocation
// entry point passes one that lives in static device memory, large enough
// for the request count, so nothing is allocated here).
static void gather_impl(const gnnav_cache *c, const int32_t *ids_dev, int64_t n_ids, const int32_t *n_dev,
                        void *out_dev, int64_t ld_out, int64_t *counts_dev, hipStream_t s,
                        hipEvent_t copy_after = nullptr, GatherWs *fixed = nullptr) {
    GNNAV_CHECK(c && counts_dev, GNNAV_E_INVALID, "NULL cache or counts");
    GNNAV_CHECK(n_ids >= 0 && n_ids < INT32_MAX, GNNAV_E_INVALID, "n_ids outside [0, INT32_MAX)");
    GNNAV_CHECK(n_ids == 0 || (ids_dev && out_dev), GNNAV_E_INVALID, "NULL ids or out");
    GNNAV_CHECK(ld_out >= c->d, GNNAV_E_INVALID, "ld_out < d");
    GNNAV_CHECK((ld_out * c->elt) % 16 == 0 && aligned16(out_dev), GNNAV_E_INVALID,
                "out rows must be 16-byte aligned");
    auto *cc = const_cast<gnnav_cache *>(c);
    // A cache that updates itself is shared mutable state: gathers on any
    // stream are ordered one after another, in call order, through an event.
    const bool dynamic = cc->ring_n > 0;
    std::unique_lock<std::mutex> upd_lock(cc->upd_mu, std::defer_lock);
    if (dynamic) {
        upd_lock.lock();
        if (cc->upd_recorded) GNNAV_HIP(hipStreamWaitEvent(s, cc->upd_done, 0));
    }
    GatherWs *w = fixed;
    if (!w) {
        w = gather_ws(cc, s);
        w->dev_counts.ensure(2 * sizeof(int32_t), s);
        w->hit_list.ensure(std::max<int64_t>(n_ids, 1) * sizeof(int2), s);
        w->miss_list.ensure(std::max<int64_t>(n_ids, 1) * sizeof(int2), s);
        w->scan.ensure(n_ids, s);
    }
    GatherArgs a{ids_dev, n_ids, n_dev, c->slot_map.as<int32_t>(), c->n, c->cache_rows.p, c->store_ptr,
                 c->ld * c->elt, c->store_pitch, out_dev, ld_out * c->elt, c->d * c->elt, counts_dev, w->dev_counts.as<int32_t>(),
                 w->hit_list.as<int2>(), w->miss_list.as<int2>(), &w->scan, cc->link_wgs};
    launch_classify(a, s);
    if (copy_after) GNNAV_HIP(hipStreamWaitEvent(s, copy_after, 0));
    if (n_ids > 0) launch_gather_rows(a, s);
    if (dynamic) {
        if (cc->policy == GNNAV_POLICY_LRU)
            launch_lru_update(a,
                              LruState{cc->ring_lo, cc->ring_n, cc->lru_order.as<int32_t>(),
                                       cc->lru_part.as<int32_t>(), cc->lru_stamp.as<uint32_t>(),
                                       cc->lru_ctl.as<uint32_t>(), &cc->lru_scan},
                              cc->owner.as<int32_t>(), cc->slot_map.as<int32_t>(), cc->cache_rows.p, s);
        else
            launch_fifo_update(a, cc->ring_lo, cc->ring_n, cc->owner.as<int32_t>(), cc->slot_map.as<int32_t>(),
                               cc->ring_ptr.as<int32_t>(), &cc->ring_parity, cc->cache_rows.p, s);
        GNNAV_HIP(hipEventRecord(cc->upd_done, s));
        cc->upd_recorded = true;
    }
}

extern "C" gnnav_status gnnav_gather(const gnnav_cache *c, const int32_t *ids_dev, int64_t n_ids, void *out_dev,
                                     int64_t ld_out, int64_t *counts_dev, void *stream) {
    return guarded([&] { gather_impl(c, ids_dev, n_ids, nullptr, out_dev, ld_out, counts_dev, (hipStream_t)stream); });
}

extern "C" gnnav_status gnnav_gather_n(const gnnav_cache *c, const int32_t *ids_dev, const int32_t *n_ids_dev,
                                       int64_t n_ids_max, void *out_dev, int64_t ld_out, int64_t *counts_dev,
                                       void *stream) {
    return guarded([&] {
        GNNAV_CHECK(n_ids_dev, GNNAV_E_INVALID, "n_ids_dev is NULL");
        gather_impl(c, ids_dev, n_ids_max, n_ids_dev, out_dev, ld_out, counts_dev, (hipStream_t)stream);
    });
}

extern "C" gnnav_status gnnav_gather_n_after(const gnnav_cache *c, const int32_t *ids_dev, const int32_t *n_ids_dev,
                                             int64_t n_ids_max, void *out_dev, int64_t ld_out, int64_t *counts_dev,
                                             void *copy_after_event, void *stream) {
    return guarded([&] {
        GNNAV_CHECK(n_ids_dev, GNNAV_E_INVALID, "n_ids_dev is NULL");
        gather_impl(c, ids_dev, n_ids_max, n_ids_dev, out_dev, ld_out, counts_dev, (hipStream_t)stream,
                    (hipEvent_t)copy_after_event);
    });
}

// --------------------------------------------- gather without allocation
// gnnav_gather_noalloc keeps its workspace -- hit and miss lists, the two
// device counts, the classification scan's ticket and tile records -- in
// `scratch`, a static device array (each device holds its own copy until the
// process ends).  Nothing in it needs clearing between calls: the lists and
// counts are written before they are read, the ticket returns to zero at the
// end of every scan launch, and tile records carry the call's epoch (the
// array starts zeroed, and epoch 0 is never used).
namespace {
constexpr int64_t kNoAllocMaxIds = int64_t(1) << 20;
constexpr size_t kNaListBytes = (size_t)kNoAllocMaxIds * sizeof(int2);
constexpr size_t kNaRecBytes = (size_t)(kNoAllocMaxIds / kScanTile) * kRecWords * sizeof(uint64_t);
constexpr size_t kNaHit = 0, kNaMiss = kNaListBytes, kNaCounts = 2 * kNaListBytes, kNaCtl = kNaCounts + 256,
                 kNaSums = kNaCtl + 256, kNaPrefix = kNaSums + kNaRecBytes, kNaBytes = kNaPrefix + kNaRecBytes;
static_assert(kNoAllocMaxIds % kScanTile == 0, "whole scan tiles");
}  // namespace

static __device__ __align__(256) unsigned char scratch[kNaBytes];

namespace {
struct NoAllocWs {
    bool ready = false;
    GatherWs ws;       // its buffers point into this device's `scratch` and are never released
    std::mutex mu;     // one call at a time per device on the host side
};
NoAllocWs g_noalloc[kMaxDevices];

// This device's workspace view; its address comes from hipGetSymbolAddress
// on the first call on the device (with that device current).
NoAllocWs &noalloc_ws() {
    const int dev = current_device();
    NoAllocWs &na = g_noalloc[dev];
    std::lock_guard<std::mutex> lk(g_err_mu);
    if (!na.ready) {
        void *ptr = nullptr;
        GNNAV_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
        GNNAV_CHECK(ptr != nullptr, GNNAV_E_DEVICE, "no device address for the static workspace");
        char *base = (char *)ptr;
        auto view = [&](DevBuf &b, size_t off, size_t bytes) {
            b.p = base + off;
            b.bytes = bytes;
        };
        view(na.ws.hit_list, kNaHit, kNaListBytes);
        view(na.ws.miss_list, kNaMiss, kNaListBytes);
        view(na.ws.dev_counts, kNaCounts, 256);
        view(na.ws.scan.ctl, kNaCtl, 256);
        view(na.ws.scan.sums, kNaSums, kNaRecBytes);
        view(na.ws.scan.prefix, kNaPrefix, kNaRecBytes);
        na.ws.scan.tiles = kNoAllocMaxIds / kScanTile;
        na.ready = true;
    }
    return na;
}
}  // namespace

extern "C" gnnav_status gnnav_gather_noalloc(const gnnav_cache *c, const int32_t *ids_dev, int64_t n_ids,
                                             void *out_dev, int64_t ld_out, int64_t *counts_dev, void *stream) {
    return guarded([&] {
        GNNAV_CHECK(n_ids <= kNoAllocMaxIds, GNNAV_E_CAPACITY,
                    "gnnav_gather_noalloc takes at most " + std::to_string(kNoAllocMaxIds) + " ids per call, got " +
                        std::to_string(n_ids));
        NoAllocWs &na = noalloc_ws();
        std::lock_guard<std::mutex> lk(na.mu);
        TimersOff quiet;   // per-kernel timing would create event objects
        gather_impl(c, ids_dev, n_ids, nullptr, out_dev, ld_out, counts_dev, (hipStream_t)stream, nullptr, &na.ws);
    });
}

// ------------------------------------------------------------------- SAGE
static int64_t padded_ld(int64_t d, int64_t elt) { return (d * elt + 15) / 16 * 16 / elt; }

extern "C" gnnav_status gnnav_aggregate_mean(const int32_t *indptr_dev, const int32_t *indices_dev, int64_t n_dst,
                                             const void *x_dev, int64_t ld_x, int64_t d, gnnav_dtype dt,
                                             void *out_dev, int64_t ld_out, void *stream) {
    return guarded([&] {
        GNNAV_CHECK(dt == GNNAV_F32 || dt == GNNAV_BF16, GNNAV_E_INVALID, "bad dtype");
        GNNAV_CHECK(n_dst >= 0 && d > 0, GNNAV_E_INVALID, "n_dst < 0 or d <= 0");
        GNNAV_CHECK(n_dst == 0 || (indptr_dev && indices_dev && x_dev && out_dev), GNNAV_E_INVALID,
                    "NULL argument");
        const int64_t elt = dt == GNNAV_BF16 ? 2 : 4;
        GNNAV_CHECK(ld_x >= d && ld_out >= d, GNNAV_E_INVALID, "stride below d");
        GNNAV_CHECK((ld_x * elt) % 16 == 0 && (ld_out * elt) % 16 == 0 && aligned16(x_dev) && aligned16(out_dev),
                    GNNAV_E_INVALID, "rows must be 16-byte aligned");
        launch_aggregate_mean(indptr_dev, indices_dev, n_dst, nullptr, x_dev, ld_x, d, dt == GNNAV_BF16, out_dev,
                              ld_out, (hipStream_t)stream);
    });
}

extern "C" int32_t gnnav_combine_kernel(int64_t m, int64_t d_out, gnnav_dtype dt) {
    if ((dt != GNNAV_F32 && dt != GNNAV_BF16) || m <= 0 || d_out <= 0) return -1;
    return combine_kernel_kind(m, d_out, dt == GNNAV_BF16);
}

extern "C" gnnav_status gnnav_combine(const void *self_dev, int64_t ld_self, const void *agg_dev, int64_t ld_agg,
                                      int64_t m, int64_t d_in, const void *w_dev, int64_t d_out, gnnav_dtype dt,
                                      int32_t relu, int32_t out_bf16, void *out_dev, int64_t ld_out,
                                      void *stream) {
    return guarded([&] {
        GNNAV_CHECK(dt == GNNAV_F32 || dt == GNNAV_BF16, GNNAV_E_INVALID, "bad dtype");
        GNNAV_CHECK(m >= 0 && d_in > 0 && d_out > 0, GNNAV_E_INVALID, "bad sizes");
        GNNAV_CHECK(m == 0 || (self_dev && agg_dev && w_dev && out_dev), GNNAV_E_INVALID, "NULL argument");
        GNNAV_CHECK(!(dt == GNNAV_F32 && out_bf16), GNNAV_E_INVALID, "bf16 output needs bf16 operands");
        const int64_t elt = dt == GNNAV_BF16 ? 2 : 4;
        GNNAV_CHECK(ld_self >= d_in && ld_agg >= d_in && ld_out >= d_out, GNNAV_E_INVALID, "stride too small");
        GNNAV_CHECK((ld_self * elt) % 16 == 0 && (ld_agg * elt) % 16 == 0 && aligned16(self_dev) &&
                        aligned16(agg_dev),
                    GNNAV_E_INVALID, "operand rows must be 16-byte aligned");
        launch_combine(self_dev, ld_self, agg_dev, ld_agg, m, nullptr, d_in, w_dev, d_out, dt == GNNAV_BF16,
                       relu != 0, out_bf16 != 0, out_dev, ld_out, (hipStream_t)stream);
    });
}

// Row counts of a block: exact host sizes after gnnav_sample /
// gnnav_blocks_sync; otherwise the kernels read them from device memory and
// grids and buffers follow the Eq. 12 bounds of the sample.
struct BlockRows {
    const gnnav_blocks *b;
    // destination rows of block hb (F_(hb-1)); hb = L + 1 gives |F_L|
    int64_t rows(int hb) const { return b->host_sizes ? b->n_h[hb - 1] : b->nb[hb - 1]; }
    const int32_t *rows_dev(int hb) const {
        return b->host_sizes ? nullptr : b->sizes.as<int32_t>() + kSizeN + hb - 1;
    }
    int64_t edges(int hb) const { return b->host_sizes ? b->e_h[hb] : b->eb[hb]; }
    const int32_t *edges_dev(int hb) const { return b->sizes.as<int32_t>() + kSizeE + hb; }
};

static const char *kAggLabel[] = {"aggregate_mean.l1", "aggregate_mean.l2", "aggregate_mean.l3", "aggregate_mean.l4+"};
static const char *kGemmLabel[] = {"combine_gemm.l1", "combine_gemm.l2", "combine_gemm.l3", "combine_gemm.l4+"};

static void check_forward_args(const gnnav_blocks *b, const void *x_dev, int64_t ld_x, const void *const *W_dev,
                               const int32_t *dims, int32_t n_layers, gnnav_dtype dt, const float *logits_dev,
                               int64_t ld_out) {
    GNNAV_CHECK(b && W_dev && dims && logits_dev, GNNAV_E_INVALID, "NULL argument");
    GNNAV_CHECK(n_layers == b->L && n_layers >= 1, GNNAV_E_INVALID, "n_layers differs from the sampled hops");
    GNNAV_CHECK(dt == GNNAV_F32 || dt == GNNAV_BF16, GNNAV_E_INVALID, "bad dtype");
    const int L = n_layers;
    for (int l = 0; l <= L; ++l) GNNAV_CHECK(dims[l] > 0, GNNAV_E_INVALID, "dims must be positive");
    for (int l = 0; l < L; ++l) GNNAV_CHECK(W_dev[l], GNNAV_E_INVALID, "NULL weight");
    GNNAV_CHECK(ld_out >= dims[L], GNNAV_E_INVALID, "ld_out < dims[L]");
    const int64_t elt = dt == GNNAV_BF16 ? 2 : 4;
    GNNAV_CHECK(ld_x >= dims[0] && (ld_x * elt) % 16 == 0 && aligned16(x_dev), GNNAV_E_INVALID,
                "x rows must be 16-byte aligned with ld_x >= dims[0]");
}

// The L-layer forward.  keep: every layer's aggregate and hidden output get
// a buffer of their own (read again by the backward); otherwise one
// aggregate buffer and two ping-pong hidden buffers are reused.
static void forward_impl(gnnav_blocks *b, const void *x_dev, int64_t ld_x, const void *const *W_dev,
                         const int32_t *dims, int L, bool bf, float *logits_dev, int64_t ld_out, bool keep,
                         hipStream_t s) {
    const int64_t elt = bf ? 2 : 4;
    const BlockRows br{b};
    if (!keep) {
        int64_t agg_bytes = 1, hid_bytes = 1;
        for (int l = 1; l <= L; ++l) {
            const int64_t rows = br.rows(L - l + 1);
            agg_bytes = std::max(agg_bytes, rows * padded_ld(dims[l - 1], elt) * elt);
            if (l < L) hid_bytes = std::max(hid_bytes, rows * padded_ld(dims[l], elt) * elt);
        }
        b->agg.ensure(agg_bytes, s);
        if (L > 1) {
            b->hid[0].ensure(hid_bytes, s);
            b->hid[1].ensure(hid_bytes, s);
        }
    }
    const void *x = x_dev;
    int64_t ldx = ld_x;
    for (int l = 1; l <= L; ++l) {
        const int tag = l < 4 ? l - 1 : 3;
        const int hb = L - l + 1;
        const int64_t rows = br.rows(hb);
        const int32_t *rdev = br.rows_dev(hb);
        const int64_t din = dims[l - 1], dout = dims[l];
        const int64_t lda = padded_ld(din, elt);
        void *agg = b->agg.p;
        if (keep) {
            b->act_agg[l - 1].ensure(std::max<int64_t>(rows, 1) * lda * elt, s);
            agg = b->act_agg[l - 1].p;
        }
        launch_aggregate_mean(b->indptr[hb - 1].as<int32_t>(), b->indices[hb - 1].as<int32_t>(), rows, rdev, x, ldx,
                              din, bf, agg, lda, s, kAggLabel[tag]);
        if (l < L) {
            const int64_t ldh = padded_ld(dout, elt);
            void *h = b->hid[l & 1].p;
            if (keep) {
                b->act_h[l - 1].ensure(std::max<int64_t>(rows, 1) * ldh * elt, s);
                h = b->act_h[l - 1].p;
            }
            launch_combine(x, ldx, agg, lda, rows, rdev, din, W_dev[l - 1], dout, bf, true, bf, h, ldh, s,
                           kGemmLabel[tag]);
            x = h;
            ldx = ldh;
        } else {
            launch_combine(x, ldx, agg, lda, rows, rdev, din, W_dev[l - 1], dout, bf, false, false, logits_dev,
                           ld_out, s, kGemmLabel[tag]);
        }
    }
}

extern "C" gnnav_status gnnav_sage_forward(gnnav_blocks *b, const void *x_dev, int64_t ld_x,
                                           const void *const *W_dev, const int32_t *dims, int32_t n_layers,
                                           gnnav_dtype dt, float *logits_dev, int64_t ld_out, void *stream) {
    return guarded([&] {
        check_forward_args(b, x_dev, ld_x, W_dev, dims, n_layers, dt, logits_dev, ld_out);
        forward_impl(b, x_dev, ld_x, W_dev, dims, n_layers, dt == GNNAV_BF16, logits_dev, ld_out, false,
                     (hipStream_t)stream);
    });
}

// ------------------------------------------------------------- training
static const char *kWgradLabel[] = {"wgrad.l1", "wgrad.l2", "wgrad.l3", "wgrad.l4+"};
static const char *kBwdGemmLabel[] = {"bwd_gemm.l1", "bwd_gemm.l2", "bwd_gemm.l3", "bwd_gemm.l4+"};
static const char *kAggTLabel[] = {"aggregate_mean_t.l1", "aggregate_mean_t.l2", "aggregate_mean_t.l3",
                                   "aggregate_mean_t.l4+"};
static const char *kCscLabel[] = {"csc_build.l1", "csc_build.l2", "csc_build.l3", "csc_build.l4+"};

extern "C" gnnav_status gnnav_sage_train_step(gnnav_blocks *b, const float *x_dev, int64_t ld_x, float *const *W_dev,
                                              const int32_t *dims, int32_t n_layers, const int32_t *labels_dev,
                                              float lr, float *logits_dev, int64_t ld_out, float *loss_dev,
                                              float *const *dW_dev, void *stream) {
    return guarded([&] {
        check_forward_args(b, x_dev, ld_x, (const void *const *)W_dev, dims, n_layers, GNNAV_F32, logits_dev, ld_out);
        GNNAV_CHECK(labels_dev && loss_dev, GNNAV_E_INVALID, "NULL labels or loss");
        GNNAV_CHECK(std::isfinite(lr), GNNAV_E_INVALID, "lr is not finite");
        const int L = n_layers;
        hipStream_t s = (hipStream_t)stream;
        forward_impl(b, x_dev, ld_x, (const void *const *)W_dev, dims, L, false, logits_dev, ld_out, true, s);
        const BlockRows br{b};
        auto ld4 = [](int64_t d) { return padded_ld(d, 4); };
        // dZ of the last layer: rows F_0
        {
            const int64_t n0 = br.rows(1);
            b->dz[L & 1].ensure(std::max<int64_t>(n0, 1) * ld4(dims[L]) * 4, s);
            b->row_loss.ensure(std::max<int64_t>(n0, 1) * 4, s);
            launch_softmax_xent(logits_dev, ld_out, n0, br.rows_dev(1), dims[L], b->nodes.as<int32_t>(), labels_dev,
                                b->dz[L & 1].as<float>(), ld4(dims[L]), b->row_loss.as<float>(), loss_dev, s);
        }
        for (int l = L; l >= 1; --l) {
            const int tag = l < 4 ? l - 1 : 3;
            const int hb = L - l + 1;
            const int64_t n_dst = br.rows(hb), n_src = br.rows(hb + 1);
            const int32_t *n_dst_dev = br.rows_dev(hb), *n_src_dev = br.rows_dev(hb + 1);
            const int64_t din = dims[l - 1], dout = dims[l];
            const float *X = l == 1 ? x_dev : b->act_h[l - 2].as<float>();
            const int64_t ldx = l == 1 ? ld_x : ld4(din);
            const float *G = b->dz[l & 1].as<float>();
            const int64_t ldg = ld4(dout);
            const float *W = W_dev[l - 1];
            if (l > 1) {
                // gradient of the layer's input: self part and aggregate part
                b->dself.ensure(std::max<int64_t>(n_dst, 1) * ld4(din) * 4, s);
                b->dagg.ensure(std::max<int64_t>(n_dst, 1) * ld4(din) * 4, s);
                launch_matmul_bt(G, ldg, n_dst, n_dst_dev, dout, W, dout, din, b->dself.as<float>(), ld4(din), s,
                                 kBwdGemmLabel[tag]);
                launch_matmul_bt(G, ldg, n_dst, n_dst_dev, dout, W + din * dout, dout, din, b->dagg.as<float>(),
                                 ld4(din), s, kBwdGemmLabel[tag]);
                b->csc.build(b->indptr[hb - 1].as<int32_t>(), b->indices[hb - 1].as<int32_t>(), n_dst, n_dst_dev,
                             br.edges_dev(hb), br.edges(hb), n_src, b->scan, s, kCscLabel[tag]);
                b->dz[(l - 1) & 1].ensure(std::max<int64_t>(n_src, 1) * ld4(din) * 4, s);
                launch_aggregate_t(b->csc, b->indptr[hb - 1].as<int32_t>(), n_src, n_src_dev, n_dst, n_dst_dev,
                                   b->dagg.as<float>(), ld4(din), b->dself.as<float>(), ld4(din), X, ldx, din,
                                   b->dz[(l - 1) & 1].as<float>(), ld4(din), s, kAggTLabel[tag]);
            }
            // dW_l = [X[0:n_dst] | agg]^T dZ_l, then W_l -= lr * dW_l
            launch_wgrad(X, ldx, b->act_agg[l - 1].as<float>(), ld4(din), n_dst, n_dst_dev, din, G, ldg, dout,
                         b->wpart, dW_dev ? dW_dev[l - 1] : nullptr, W_dev[l - 1], lr, s, kWgradLabel[tag]);
        }
    });
}

// Stand-alone entry points of the backward kernels.  They share one
// process-wide workspace; an event recorded after each call orders the next
// one after it, whichever stream it uses.
namespace {
struct TrainWs {
    std::mutex mu;
    CscWorkspace csc;
    ScanState scan;
    DevBuf part, count;
    hipEvent_t last_use = nullptr;
};
TrainWs g_train;

template <class F>
void with_train_ws(hipStream_t s, F &&f) {
    std::lock_guard<std::mutex> lk(g_train.mu);
    if (!g_train.last_use) GNNAV_HIP(hipEventCreateWithFlags(&g_train.last_use, hipEventDisableTiming));
    GNNAV_HIP(hipStreamWaitEvent(s, g_train.last_use, 0));
    f(g_train);
    GNNAV_HIP(hipEventRecord(g_train.last_use, s));
}
}  // namespace

extern "C" gnnav_status gnnav_softmax_xent(const float *logits_dev, int64_t ld, int64_t n, int64_t n_classes,
                                           const int32_t *labels_dev, float *dz_dev, int64_t ld_dz, float *loss_dev,
                                           void *stream) {
    return guarded([&] {
        GNNAV_CHECK(n >= 0 && n_classes > 0, GNNAV_E_INVALID, "n < 0 or n_classes <= 0");
        GNNAV_CHECK(loss_dev && (n == 0 || (logits_dev && labels_dev && dz_dev)), GNNAV_E_INVALID, "NULL argument");
        GNNAV_CHECK(ld >= n_classes && ld_dz >= n_classes, GNNAV_E_INVALID, "stride below n_classes");
        hipStream_t s = (hipStream_t)stream;
        with_train_ws(s, [&](TrainWs &w) {
            w.part.ensure(std::max<int64_t>(n, 1) * sizeof(float), s);
            launch_softmax_xent(logits_dev, ld, n, nullptr, n_classes, nullptr, labels_dev, dz_dev, ld_dz,
                                w.part.as<float>(), loss_dev, s);
        });
    });
}

extern "C" gnnav_status gnnav_aggregate_mean_backward(const int32_t *indptr_dev, const int32_t *indices_dev,
                                                      int64_t n_dst, int64_t n_src, const float *dagg_dev,
                                                      int64_t ld_dagg, const float *dself_dev, int64_t ld_dself,
                                                      const float *mask_dev, int64_t ld_mask, int64_t d,
                                                      float *out_dev, int64_t ld_out, void *stream) {
    return guarded([&] {
        GNNAV_CHECK(n_dst >= 0 && n_src >= 0 && d > 0, GNNAV_E_INVALID, "negative size or d <= 0");
        GNNAV_CHECK(n_src < INT32_MAX && n_dst < INT32_MAX, GNNAV_E_INVALID, "sizes beyond int32");
        GNNAV_CHECK(n_dst == 0 || (indptr_dev && indices_dev && dagg_dev), GNNAV_E_INVALID, "NULL block or dagg");
        GNNAV_CHECK(n_src == 0 || out_dev, GNNAV_E_INVALID, "NULL out");
        auto rows_ok = [&](const float *p, int64_t ld) {
            return p == nullptr || (ld >= d && ld % 4 == 0 && aligned16(p));
        };
        GNNAV_CHECK(rows_ok(dagg_dev, ld_dagg) && rows_ok(dself_dev, ld_dself) && rows_ok(mask_dev, ld_mask) &&
                        rows_ok(out_dev, ld_out),
                    GNNAV_E_INVALID, "rows must be 16-byte aligned with ld >= d");
        GNNAV_CHECK(dself_dev == nullptr || n_dst <= n_src, GNNAV_E_INVALID, "self term needs n_dst <= n_src");
        if (n_src == 0) return;
        hipStream_t s = (hipStream_t)stream;
        int32_t n_edges = 0;
        if (n_dst > 0)
            GNNAV_HIP(hipMemcpy(&n_edges, indptr_dev + n_dst, sizeof(int32_t), hipMemcpyDeviceToHost));
        with_train_ws(s, [&](TrainWs &w) {
            w.count.ensure(sizeof(int32_t), s);
            launch_fill_i32(w.count.as<int32_t>(), n_edges, 1, s);
            w.csc.build(indptr_dev, indices_dev, n_dst, nullptr, w.count.as<int32_t>(), n_edges, n_src, w.scan, s,
                        "csc_build");
            launch_aggregate_t(w.csc, indptr_dev, n_src, nullptr, dself_dev ? n_dst : 0, nullptr, dagg_dev, ld_dagg,
                               dself_dev, ld_dself, mask_dev, ld_mask, d, out_dev, ld_out, s, "aggregate_mean_t");
        });
    });
}

extern "C" gnnav_status gnnav_weight_grad(const float *self_dev, int64_t ld_self, const float *agg_dev,
                                          int64_t ld_agg, int64_t m, int64_t d_in, const float *dz_dev,
                                          int64_t ld_dz, int64_t d_out, float *dw_dev, void *stream) {
    return guarded([&] {
        GNNAV_CHECK(m >= 0 && d_in > 0 && d_out > 0, GNNAV_E_INVALID, "m < 0 or d <= 0");
        GNNAV_CHECK(dw_dev && (m == 0 || (self_dev && agg_dev && dz_dev)), GNNAV_E_INVALID, "NULL argument");
        GNNAV_CHECK(ld_self >= d_in && ld_agg >= d_in && ld_dz >= d_out, GNNAV_E_INVALID, "stride below width");
        GNNAV_CHECK(ld_self % 4 == 0 && ld_agg % 4 == 0 && ld_dz % 4 == 0 &&
                        (m == 0 || (aligned16(self_dev) && aligned16(agg_dev) && aligned16(dz_dev))),
                    GNNAV_E_INVALID, "rows must be 16-byte aligned");
        hipStream_t s = (hipStream_t)stream;
        with_train_ws(s, [&](TrainWs &w) {
            launch_wgrad(self_dev, ld_self, agg_dev, ld_agg, m, nullptr, d_in, dz_dev, ld_dz, d_out, w.part, dw_dev,
                         nullptr, 0.0f, s, "wgrad");
        });
    });
}
