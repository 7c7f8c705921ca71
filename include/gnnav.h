/* gnnav.h -- C ABI of the MI355X sampled mini-batch step for GraphSAGE-style
 * training, as decomposed by GNNavigator (DAC'24, arXiv 2404.09544).
 *
 * One mini-batch (Algorithm 1, Section 2.1, forward part) is:
 *   gnnav_sample        Eq. 2 node-wise fanout sampling plus the per-hop
 *                       union (dedup/relabel) of the sampled frontier;
 *   gnnav_gather        the device-cache step of Section 3.2 ("Transmission
 *                       strategies"): cached rows read from HBM, the rest
 *                       read from the host store over the host-device link;
 *   gnnav_sage_forward  Eq. 1 per layer: mean Aggregate over sampled
 *                       neighbours, then the SAGE Combine (one GEMM).
 * gnnav_build_csr and gnnav_build_cache are one-time set-up.
 *
 * Conventions shared by every entry point:
 *   - Status codes only; no C++ exception crosses this boundary.  A failing
 *     call leaves a message readable through gnnav_last_error() (per thread,
 *     valid until that thread's next gnnav_* call).
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *   - "device" pointers are HBM addresses on the current HIP device;
 *     "host" pointers are ordinary process memory.  Row-major everywhere.
 *   - `ld` arguments are row strides in elements.  Feature-row strides must
 *     make every row start on a 16-byte boundary (ld * element size is a
 *     multiple of 16 and the base pointer is 16-byte aligned).
 *   - Handles are created by gnnav_build_* / gnnav_blocks_create and freed by
 *     the matching *_free, which accepts NULL.  Handles copy their inputs;
 *     callers keep ownership of every buffer they pass in.  A call that fails
 *     leaves its output handle (*out) unwritten.
 *   - Asynchronous calls (gather, aggregate, combine, forward, train step,
 *     gnnav_sample_async) report argument and allocation errors at once;
 *     a failure the device itself detects while running them (a device-wide
 *     scan whose look-back wait gave up) is counted in a per-device error
 *     word and reported as E_DEVICE by the next synchronisation point:
 *     gnnav_sync, gnnav_blocks_sync or gnnav_sample.
 */
#ifndef GNNAV_H
#define GNNAV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GNNAV_ABI_VERSION 1

typedef enum gnnav_status {
    GNNAV_OK = 0,
    GNNAV_E_INVALID = 1,   /* bad argument: null pointer, bad size, bad stride */
    GNNAV_E_RANGE = 2,     /* a node id outside [0, n) where ids must be valid */
    GNNAV_E_NOMEM = 3,     /* host, pinned or device allocation failed */
    GNNAV_E_CAPACITY = 4,  /* a size bound exceeds the 32-bit local-id range */
    GNNAV_E_DEVICE = 5     /* a HIP runtime error, or a failure the device reported
                              (gnnav_sync); its text is in last_error */
} gnnav_status;

typedef enum gnnav_dtype { GNNAV_F32 = 0, GNNAV_BF16 = 1 } gnnav_dtype;

/* gnnav_build_csr flags */
#define GNNAV_SYMMETRIZE 0x1u   /* add (v,u) for every input pair (u,v) */
#define GNNAV_OFFSETS_I64 0x2u  /* keep row offsets as int64 on the device */
/* gnnav_build_cache flags */
#define GNNAV_STORE_ON_DEVICE 0x1u /* the full feature store lives in HBM */

typedef struct gnnav_graph gnnav_graph;
typedef struct gnnav_cache gnnav_cache;
typedef struct gnnav_blocks gnnav_blocks;

/* One sampled hop h (1-based): destinations F_(h-1), sources F_h. */
typedef struct gnnav_block_view {
    int64_t n_dst;            /* |F_(h-1)| */
    int64_t n_src;            /* |F_h| */
    int64_t nnz;              /* E_h, sampled edges of this hop */
    const int32_t *indptr;    /* device, n_dst + 1: row i owns [indptr[i], indptr[i+1]) */
    const int32_t *indices;   /* device, nnz: local ids in [0, n_src) */
    const int32_t *neighbors; /* device, nnz: the same edges as global node ids */
    const int32_t *src_ids;   /* device, n_src: global ids of F_h (prefix of the node list) */
} gnnav_block_view;

/* Message of this thread's last failing call ("" if none). */
const char *gnnav_last_error(void);

/* GNNAV_ABI_VERSION of the loaded library. */
int32_t gnnav_abi_version(void);

/* Synchronisation point for asynchronous work: waits for `stream`, then
 * returns E_DEVICE if device-side work on the current device (any stream)
 * has reported a failure since the last report -- a device-wide scan (the
 * classification of gnnav_gather*, the sampler's count and dedup scans, the
 * backward's block transpose) whose look-back wait gave up, which leaves
 * that work's results unreliable.  Each failure is reported once.
 * Errors: E_DEVICE.                                                        */
gnnav_status gnnav_sync(void *stream);

/* A stream whose kernels run on one share of the device's compute units,
 * for pipelines that overlap one batch's host-link transfer with another
 * batch's sampling and computation (Eq. 4's max of the two): batches
 * enqueued on streams of different shares never share a compute unit, so
 * the host-link workgroups of one batch's gather keep their issue rate
 * while the other batch runs.  Share `part` of `parts` takes the CU-mask
 * bits i with (i / 8) mod parts == part; on MI355X the runtime deals mask
 * bits out to the eight XCDs in turn, so a share holds every parts-th
 * compute unit of every XCD.  Results of work on such a stream are those of
 * any other stream; only its speed differs (a share of the units), which
 * pays where the transfer dominates the step and costs where it does not.
 * The stream has the default priority.  The caller owns it: release it
 * with gnnav_stream_destroy.  *out is written only on success.
 * Errors: E_INVALID (NULL out, parts outside [1, 8], part outside
 * [0, parts), fewer than 8 compute units per share), E_DEVICE (the runtime
 * refused the stream).                                                     */
gnnav_status gnnav_stream_create(int32_t part, int32_t parts, void **out);

/* Waits for the work on a stream from gnnav_stream_create, then releases
 * it.  NULL is allowed.  Errors: E_DEVICE.                                  */
gnnav_status gnnav_stream_destroy(void *stream);

/* ---------------------------------------------------------------- graph ---
 * Graph G(V, E) of Algorithm 1's input, as CSR in HBM.
 * src, dst: host arrays of n_edges node ids in [0, n_nodes).  Self pairs are
 * dropped, repeated pairs kept once, and with GNNAV_SYMMETRIZE each pair is
 * stored in both directions.  Each row lists its neighbours in ascending id
 * order.  Offsets are int32 unless GNNAV_OFFSETS_I64 is set or nnz needs
 * more; column ids are int32.
 * Errors: E_INVALID (null pointers with n_edges > 0, n_nodes < 0 or
 * > INT32_MAX, out == NULL), E_RANGE (an endpoint outside [0, n_nodes)),
 * E_NOMEM, E_DEVICE.  On error *out is left unchanged.                    */
gnnav_status gnnav_build_csr(int64_t n_nodes, int64_t n_edges, const int32_t *src,
                             const int32_t *dst, uint32_t flags, gnnav_graph **out);

/* Sizes of a graph; any output pointer may be NULL. */
gnnav_status gnnav_graph_info(const gnnav_graph *g, int64_t *n_nodes, int64_t *nnz,
                              int64_t *max_degree, int32_t *offsets_i64);

/* Host copies of the CSR: row_ptr (int64, n_nodes+1 entries) and col
 * (int32, nnz entries; NULL skips it), caller-allocated.  For tests and
 * tooling.  Errors: E_INVALID (g or row_ptr NULL), E_DEVICE.              */
gnnav_status gnnav_graph_csr_host(const gnnav_graph *g, int64_t *row_ptr, int32_t *col);

void gnnav_graph_free(gnnav_graph *g);

/* ---------------------------------------------------------------- cache ---
 * Static device feature cache in front of a pinned host feature store
 * (Section 3.2, "Transmission strategies", with the cache-update policy
 * disabled and a cache ratio, as in the PaGraph template of Section 3.2 and
 * the static-cache baseline of Section 4.1).
 * feats_host: n_nodes x d row-major (n_nodes of g), float32 or bfloat16 bit
 * patterns.  The C = floor(cache_fraction * n_nodes) vertices of largest
 * degree (ties: smaller id first) get cache slots 0..C-1 in that order and
 * their rows are copied into HBM.  Every row is also copied into a pinned,
 * device-mapped host store (or an HBM store with GNNAV_STORE_ON_DEVICE).
 * Cache rows are padded with zeros to a 16-byte stride (see cache_info);
 * rows of a host store start on 128-byte boundaries, so the zero-copy reads
 * of a miss cross as few of the link's read blocks as the row allows.
 * Errors: E_INVALID (null pointers, d <= 0, cache_fraction outside [0, 1]
 * or NaN, bad dtype), E_NOMEM, E_DEVICE.  On error *out is unchanged.     */
gnnav_status gnnav_build_cache(const gnnav_graph *g, const void *feats_host, int64_t d,
                               gnnav_dtype dt, double cache_fraction, uint32_t flags,
                               gnnav_cache **out);

/* Cache geometry; any output pointer may be NULL.  ld is the padded row
 * stride in elements of the HBM cache (and of an HBM store).            */
gnnav_status gnnav_cache_info(const gnnav_cache *c, int64_t *n_cached, int64_t *d, int64_t *ld,
                              int32_t *dtype, int32_t *store_on_device);

/* Host copy of the current slot map (int32[n_nodes]: slot, or -1 if not
 * cached).  Synchronises the device.                                       */
gnnav_status gnnav_cache_slot_map_host(const gnnav_cache *c, int32_t *slot_map);

/* Host copies of the current cache contents (synchronises the device):
 * owners (int32[n_cached], vertex held in each slot) and rows
 * (n_cached x ld elements); either may be NULL.  For tests and tooling.   */
gnnav_status gnnav_cache_contents_host(const gnnav_cache *c, int32_t *owners, void *rows);

/* Number of workgroups of each later gather that copy the uncached rows
 * from the host store over the host link (zero-copy reads; Section 3.2's
 * transmission of the misses).  Default 64, which keeps the link at its
 * measured rate on MI355X.  Every one of their reads waits microseconds in
 * the memory system, and while they are queued, kernels running alongside
 * (the previous batch's compute in a pipeline) see their own memory
 * accesses slow down; a smaller count (e.g. 32) gives up about 3% of the
 * link rate for much less of that.  Results do not depend on the count.
 * Host-side setting, read when a gather is enqueued.
 * Errors: E_INVALID (NULL cache, workgroups outside [1, 4096]).            */
gnnav_status gnnav_cache_set_link_workgroups(gnnav_cache *c, int32_t workgroups);

/* Cache update policy (the last step of Section 3.2's transmission
 * abstraction: after a batch, the cache is updated by its policy; the cost
 * is Eq. 5's t_replace).  GNNAV_POLICY_STATIC (default) never changes the
 * cache.  GNNAV_POLICY_FIFO makes the last dynamic_slots cache slots a ring:
 * after each gather, the batch's misses are admitted in request order, each
 * taking the slot under the ring pointer and advancing the pointer; the
 * slot's previous vertex is evicted (unmapped unless the slot map already
 * points it at another slot); the earlier slots keep their degree-ranked
 * vertices.  A vertex requested more than once in one gather is admitted
 * once per missing request and stays mapped to the last of its slots (the
 * others hold copies of its row until the ring reaches them); request lists
 * without repeats, such as a frontier, never do this.
 * GNNAV_POLICY_LRU uses the same ring with a recency order in place of the
 * pointer (least recently used first, counted in batches: all requests of
 * one gather are one use).  After each gather the ring slots it hit move
 * behind every slot it did not touch, each group keeping its earlier
 * order; then the misses are admitted in request order as above, each
 * taking the least recently used slot, which becomes the most recent.
 * With no hit on the ring this is FIFO.  The ring holds per slot 12 bytes
 * of device state besides the row.  If the device-wide scan that reorders
 * the list gives up (E_DEVICE at the next synchronisation point), that
 * gather's update is skipped and the cache stays as it was.
 * Rows are copied from the gather's own output.  With a dynamic cache,
 * gathers on different streams run one after another in call order.  The
 * call synchronises the device and restarts the ring pointer at the ring's
 * first slot (LRU: the recency order at the slot order, lowest slot least
 * recent); the cache contents are kept.
 * Errors: E_INVALID (unknown policy, dynamic_slots outside [0, n_cached]);
 * E_NOMEM (the ring's device state; the cache is then left static).       */
#define GNNAV_POLICY_STATIC 0
#define GNNAV_POLICY_FIFO 1
#define GNNAV_POLICY_LRU 2
gnnav_status gnnav_cache_set_policy(gnnav_cache *c, int32_t policy, int64_t dynamic_slots);

void gnnav_cache_free(gnnav_cache *c);

/* --------------------------------------------------------------- sample ---
 * Blocks: device workspace that receives the sampled frontiers and hops.
 * It grows on demand and is reused across calls (no per-batch allocation
 * once it has reached the largest batch's size).                          */
gnnav_status gnnav_blocks_create(gnnav_blocks **out);
void gnnav_blocks_free(gnnav_blocks *b);

/* Eq. 2 node-wise sampling for n_hops hops plus the union of each hop.
 * seeds_dev: device int32[n_seeds], the target vertices B^0 (repeats are
 * dropped, first occurrence kept).  fanouts: host int32[n_hops]; fanouts[0]
 * applies to the seeds; k < 0 takes every neighbour.  For each node v of
 * F_(h-1) (every node, including ones reached earlier): if deg(v) <= k the
 * whole row, else k distinct neighbours by Floyd's selection whose draws
 * are Philox4x32-10 word 0 with key (lo32, hi32 of rng_seed) and counter
 * (slot j, lo32 v, hi32 v, h-1), each mapped to [0, m] as floor(x*(m+1)/2^32).
 * F_h is F_(h-1) followed by the new ids in order of first occurrence.
 * Results stay on the device in `blocks` (see gnnav_blocks_hop/_nodes);
 * they are valid until the next gnnav_sample on the same blocks.  The call
 * enqueues its kernels on `stream` and synchronises that stream once at the
 * end to publish the per-hop sizes to the host.
 * Errors: E_INVALID (null pointers, n_hops < 1 or > 16, n_seeds < 0),
 * E_CAPACITY (an Eq. 12 bound exceeds INT32_MAX; checked on the host
 * before anything is enqueued, so the blocks keep the previous sample),
 * E_RANGE (a seed outside [0, n); the blocks' contents are then unspecified
 * but reusable), E_NOMEM (the blocks then hold no sample: views and the
 * forward refuse them with E_INVALID until a sample succeeds), E_DEVICE
 * (also: a device-side failure, see gnnav_sync).                          */
gnnav_status gnnav_sample(const gnnav_graph *g, const int32_t *seeds_dev, int64_t n_seeds,
                          const int32_t *fanouts, int32_t n_hops, uint64_t rng_seed,
                          gnnav_blocks *blocks, void *stream);

/* gnnav_sample without the final synchronisation: every kernel is enqueued
 * on `stream` and the call returns at once; frontier and hop sizes stay in
 * device memory.  Later work on the same stream (gnnav_gather_n,
 * gnnav_sage_forward) reads them there.  Host-side size views
 * (gnnav_blocks_hop, n_per_hop of gnnav_blocks_nodes) need
 * gnnav_blocks_sync first.  A seed outside [0, n) is skipped and reported
 * as E_RANGE by the next gnnav_blocks_sync.  Same errors as gnnav_sample
 * otherwise (argument and capacity checks happen before anything is
 * enqueued).                                                               */
gnnav_status gnnav_sample_async(const gnnav_graph *g, const int32_t *seeds_dev, int64_t n_seeds,
                                const int32_t *fanouts, int32_t n_hops, uint64_t rng_seed,
                                gnnav_blocks *blocks, void *stream);

/* Waits for `stream` and copies the last sample's sizes to the host.
 * Errors: E_INVALID (never sampled), E_RANGE (seeds outside [0, n) were
 * skipped), E_DEVICE (a HIP error, or a device-side failure reported as by
 * gnnav_sync; the sizes are then not published).                           */
gnnav_status gnnav_blocks_sync(gnnav_blocks *b, void *stream);

/* Device view of the last sample's sizes, valid once the sample's kernels
 * have run: (*sizes_dev)[h] = |F_h| for h = 0..L and (*sizes_dev)[17 + h] =
 * E_h for h = 1..L (int32).  bounds (host int64[L+1], may be NULL) receives
 * the Eq. 12 capacity bounds the buffers were sized for.                  */
gnnav_status gnnav_blocks_device_sizes(const gnnav_blocks *b, const int32_t **sizes_dev,
                                       int64_t *bounds);

/* View of hop h (1..n_hops) of the last gnnav_sample. */
gnnav_status gnnav_blocks_hop(const gnnav_blocks *b, int32_t hop, gnnav_block_view *out);

/* All frontiers: *nodes_dev = device int32 list whose first n_per_hop[h]
 * entries are F_h; n_per_hop receives n_hops+1 sizes (host int64 array,
 * caller-allocated, may be NULL); *n_hops receives L (may be NULL).       */
gnnav_status gnnav_blocks_nodes(const gnnav_blocks *b, const int32_t **nodes_dev,
                                int64_t *n_per_hop, int32_t *n_hops);

/* --------------------------------------------------------------- gather ---
 * Section 3.2's cache step for n_ids requested vertices: out row i (device,
 * stride ld_out elements of the cache dtype) becomes the feature row of
 * ids_dev[i].  Cached vertices are copied from HBM; the rest are read from
 * the host store by zero-copy loads over the host-device link, in the same
 * launch on `stream` (a share of its workgroups, gnnav_cache_set_link_
 * workgroups).  Gathers on the same static cache from different streams may
 * overlap.  Each row
 * copies ceil(d * elt / 16) 16-byte units: the columns from d up to the
 * next 16-byte boundary are written with zeros; later columns are untouched.
 * An id outside [0, n) gives a zero row and counts as invalid.
 * counts_dev: device int64[3] receiving {hits, misses, invalid}; overwritten.
 * Asynchronous with respect to the host; a device-side failure of the
 * classification is reported by the next gnnav_sync.
 * Errors: E_INVALID (null pointers with n_ids > 0, ld_out < d, row stride
 * not a multiple of 16 bytes or out_dev not 16-byte aligned), E_NOMEM,
 * E_DEVICE.                                                               */
gnnav_status gnnav_gather(const gnnav_cache *c, const int32_t *ids_dev, int64_t n_ids,
                          void *out_dev, int64_t ld_out, int64_t *counts_dev, void *stream);

/* gnnav_gather with the request count read from device memory (e.g. the
 * |F_L| entry of gnnav_blocks_device_sizes) when the work runs.  out_dev
 * must hold n_ids_max rows; counts as gnnav_gather.  Calls on different
 * streams may overlap: each stream gets its own scratch inside the cache.
 * Errors as gnnav_gather, plus E_INVALID for a NULL n_ids_dev.            */
gnnav_status gnnav_gather_n(const gnnav_cache *c, const int32_t *ids_dev, const int32_t *n_ids_dev,
                            int64_t n_ids_max, void *out_dev, int64_t ld_out, int64_t *counts_dev,
                            void *stream);

/* gnnav_gather_n whose row copies (not the classification) wait for
 * copy_after_event (a hipEvent_t, or NULL for no wait) to complete: a
 * pipeline passes the previous batch's gather event, so transfers over the
 * host link run one after another while each batch's classification runs
 * ahead.  Same results and errors as gnnav_gather_n.                      */
gnnav_status gnnav_gather_n_after(const gnnav_cache *c, const int32_t *ids_dev,
                                  const int32_t *n_ids_dev, int64_t n_ids_max, void *out_dev,
                                  int64_t ld_out, int64_t *counts_dev, void *copy_after_event,
                                  void *stream);

/* gnnav_gather for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same results as gnnav_gather (any update policy) for at most
 * 1,048,576 ids, with no hipMalloc, hipFree or other allocation.  Its
 * workspace (hit and miss lists, counts, the classification scan's ticket
 * and tile records; about 16.02 MiB per device) is a static device array
 * that each device the library runs on holds until the process ends.  Every
 * call on a device shares that device's array: calls whose work overlaps on
 * one device race (this one enqueues its work after the previous call's on
 * the same stream; across streams the caller must order them).  The array
 * keeps the last call's contents; nothing in it needs clearing.  Per-kernel
 * profiling records nothing for these calls.
 * Errors: E_CAPACITY (n_ids above 1,048,576, before any work), otherwise as
 * gnnav_gather without E_NOMEM.                                            */
gnnav_status gnnav_gather_noalloc(const gnnav_cache *c, const int32_t *ids_dev, int64_t n_ids,
                                  void *out_dev, int64_t ld_out, int64_t *counts_dev, void *stream);

/* ------------------------------------------------------- SAGE, per layer ---
 * Eq. 1 Aggregate, GraphSAGE mean: for each destination row i < n_dst,
 * out[i] = (1/cnt_i) * sum over p in [indptr[i], indptr[i+1]) of
 * x[indices[p]], or zeros when the row is empty.  fp32 accumulation in CSR
 * order; bf16 inputs give bf16 outputs rounded to nearest-even.  x and out
 * are device matrices with strides ld_x, ld_out (16-byte row alignment);
 * columns from d up to the next 16-byte boundary of out are written with
 * zeros.  indptr/indices are device int32 (a block of gnnav_sample or any
 * CSR whose indices are valid rows of x).
 * Errors: E_INVALID (null pointers with n_dst > 0, d <= 0, strides < d or
 * misaligned), E_DEVICE.  Asynchronous.                                   */
gnnav_status gnnav_aggregate_mean(const int32_t *indptr_dev, const int32_t *indices_dev,
                                  int64_t n_dst, const void *x_dev, int64_t ld_x, int64_t d,
                                  gnnav_dtype dt, void *out_dev, int64_t ld_out, void *stream);

/* Eq. 1 Combine for SAGE: out = act(self * W[0:d_in] + agg * W[d_in:2*d_in])
 * for m rows, with W row-major [2*d_in, d_out] (device), self and agg
 * device [m x d_in] with strides ld_self, ld_agg.  act is ReLU when relu is
 * nonzero.  dt = F32: fp32 operands and output, fp32-accurate products: fp32
 * MFMA for few rows, otherwise both operands cut into three bf16 parts on
 * the bf16 matrix cores (six part products per fp32 product, accumulated in
 * fp32; see gnnav_combine_kernel).  dt = BF16:
 * bf16 operands, fp32 accumulation, output bf16 (nearest-even) when
 * out_bf16 is nonzero, else fp32.  The concatenation [self | agg] is never
 * formed.  self and agg rows start 16-byte aligned; out needs only its
 * element's alignment (aligned rows are stored 16 bytes at a time).
 * Errors: E_INVALID (null pointers with m > 0, d_in or d_out <= 0, strides
 * too small, self or agg rows misaligned), E_DEVICE.  Asynchronous.       */
gnnav_status gnnav_combine(const void *self_dev, int64_t ld_self, const void *agg_dev,
                           int64_t ld_agg, int64_t m, int64_t d_in, const void *w_dev,
                           int64_t d_out, gnnav_dtype dt, int32_t relu, int32_t out_bf16,
                           void *out_dev, int64_t ld_out, void *stream);

/* Which kernel a combine of m rows (the row count, or its bound when the
 * count is read on the device) and d_out output columns runs, the one
 * gnnav_combine, gnnav_sage_forward and gnnav_sage_train_step launch:
 * GNNAV_COMBINE_SKINNY: few rows, fp32 or bf16 MFMA as the dtype;
 * GNNAV_COMBINE_RING: bf16 MFMA; GNNAV_COMBINE_SPLIT: fp32 through the
 * three-way bf16 split, six bf16 MFMA products per fp32 product.  Host only,
 * no device work; -1 for dt other than F32/BF16 or sizes <= 0.           */
enum { GNNAV_COMBINE_SKINNY = 0, GNNAV_COMBINE_RING = 1, GNNAV_COMBINE_SPLIT = 2 };
int32_t gnnav_combine_kernel(int64_t m, int64_t d_out, gnnav_dtype dt);

/* ---------------------------------------------------------- SAGE forward ---
 * Algorithm 1, its per-layer aggregate/combine loop (forward only): n_layers = L of the last
 * gnnav_sample on `b`.  Layer l (1-based) runs on hop b = L-l+1:
 * destinations F_(b-1), sources F_b; it aggregates (mean) and combines with
 * W_dev[l-1] (device, row-major [2*dims[l-1], dims[l]]), applies ReLU for
 * l < L.  x_dev holds the n_L input rows of F_L (stride ld_x, dims[0]
 * used), e.g. the output of gnnav_gather on F_L.  logits_dev receives the
 * |F_0| x dims[L] fp32 result (stride ld_out).  dt = BF16 keeps features,
 * weights, aggregates and hidden layers in bfloat16 (fp32 accumulation);
 * the logits stay fp32.  Intermediate buffers live in `b` and are reused.
 * After gnnav_sample_async (no gnnav_blocks_sync) the row counts are read
 * from device memory and logits_dev must hold min(n_seeds, n) rows.
 * Errors: E_INVALID (null pointers, n_layers differs from the sampled
 * hops, dims <= 0, strides), E_NOMEM, E_DEVICE.  Asynchronous.            */
gnnav_status gnnav_sage_forward(gnnav_blocks *b, const void *x_dev, int64_t ld_x,
                                const void *const *W_dev, const int32_t *dims, int32_t n_layers,
                                gnnav_dtype dt, float *logits_dev, int64_t ld_out, void *stream);

/* -------------------------------------------------------------- training ---
 * The rest of Algorithm 1's iteration after the forward: the loss over the
 * target vertices, the backward pass through the L SAGE layers and the
 * weight update.  fp32 only.  The paper fixes neither loss nor optimiser;
 * these entry points use mean softmax cross-entropy and plain SGD.
 *
 * gnnav_sage_train_step: forward as gnnav_sage_forward (dt = F32), keeping
 * every layer's aggregate and hidden output in `b`; then
 *   loss = mean over rows i of F_0 of -log softmax(Z_L[i])[y_i], with
 *          y_i = labels_dev[F_0[i]] (labels_dev: device int32, one per
 *          graph vertex); written to loss_dev[0];
 *   dZ_L = (softmax(Z_L) - onehot(y)) / |F_0|;
 *   for l = L .. 1 (block b = L-l+1, X = H^(l-1), n = |F_(b-1)|):
 *     dW_l = [X[0:n] | Agg_l]^T dZ_l;
 *     for l > 1: dX = dZ_l W_top^T on the first n rows plus the adjoint of
 *     the mean aggregation applied to dZ_l W_bot^T (row j receives
 *     dAgg[i] / cnt_i from every sampled edge i -> j), and
 *     dZ_(l-1) = dX * [H^(l-1) > 0];
 *   W_dev[l-1] -= lr * dW_l, in place, after dZ_(l-1) has been computed.
 * Every sum runs in a fixed order (no floating-point atomics): repeated
 * calls on the same inputs give identical bits.  dW_dev: optional array of
 * L device pointers that receive dW_l (row-major [2*dims[l-1], dims[l]]);
 * NULL skips the copy.  A label outside [0, dims[L]) makes that row's loss
 * NaN (so the mean is NaN) and its gradient row zero.
 * Errors: as gnnav_sage_forward; E_INVALID also for NULL labels/loss or a
 * non-finite lr.  Asynchronous.                                           */
gnnav_status gnnav_sage_train_step(gnnav_blocks *b, const float *x_dev, int64_t ld_x,
                                   float *const *W_dev, const int32_t *dims, int32_t n_layers,
                                   const int32_t *labels_dev, float lr, float *logits_dev,
                                   int64_t ld_out, float *loss_dev, float *const *dW_dev, void *stream);

/* The backward kernels one at a time (device pointers, fp32, rows 16-byte
 * aligned; the three share one process-wide workspace, ordered across
 * streams by an event).
 *
 * gnnav_softmax_xent: loss_dev[0] = mean over the n rows of logits [n x C]
 * of the softmax cross-entropy with labels_dev[i] (device int32[n]);
 * dz_dev [n x C] = (softmax - onehot) / n.  Labels outside [0, C) as above.
 *
 * gnnav_aggregate_mean_backward: the adjoint of gnnav_aggregate_mean for a
 * block (indptr [n_dst+1], indices [E] local source ids < n_src):
 *   out[j] = mask(j) * ( sum over edges p with indices[p] = j, in edge
 *            order, of dagg[i(p)] / cnt_i  +  dself[j] if j < n_dst ),
 * for j < n_src; dself_dev and mask_dev may be NULL (no self term; no mask),
 * mask(j) zeroes the elements where mask_dev[j] <= 0.  Reads indptr[n_dst]
 * to the host (one synchronous copy).
 *
 * gnnav_weight_grad: dw_dev [2*d_in x d_out] (contiguous) =
 * [self | agg]^T dz for m rows (Eq. 1's combine, differentiated).
 * Errors: E_INVALID (null pointers, sizes, strides, alignment), E_DEVICE. */
gnnav_status gnnav_softmax_xent(const float *logits_dev, int64_t ld, int64_t n, int64_t n_classes,
                                const int32_t *labels_dev, float *dz_dev, int64_t ld_dz,
                                float *loss_dev, void *stream);
gnnav_status gnnav_aggregate_mean_backward(const int32_t *indptr_dev, const int32_t *indices_dev,
                                           int64_t n_dst, int64_t n_src, const float *dagg_dev,
                                           int64_t ld_dagg, const float *dself_dev, int64_t ld_dself,
                                           const float *mask_dev, int64_t ld_mask, int64_t d,
                                           float *out_dev, int64_t ld_out, void *stream);
gnnav_status gnnav_weight_grad(const float *self_dev, int64_t ld_self, const float *agg_dev,
                               int64_t ld_agg, int64_t m, int64_t d_in, const float *dz_dev,
                               int64_t ld_dz, int64_t d_out, float *dw_dev, void *stream);

/* -------------------------------------------------- locality-biased sampler ---
 * gnnav_sample with the neighbour-selection probability made a function of
 * data locality, p(eta) (Section 3.2, the sampler abstraction that
 * reproduces cache-aware samplers): a neighbour held in `cache` (slot map
 * >= 0) weighs eta, any other 1, and for deg(v) > k the k picks are made by
 * successive sampling without replacement with those weights (eta = 1 is
 * uniform; a large eta takes cached neighbours first).  Done as: for pick
 * j = 0..k-1 in order, with c_r cached and u_r uncached neighbours left,
 * t = floor(x * (eta*c_r + u_r) / 2^32) with x = Philox4x32-10 word 1 of
 * the counter of gnnav_sample (j, lo32 v, hi32 v, h-1); the pick is cached
 * when t < eta*c_r.  Then a uniform subset of each class by Floyd's
 * selection over the class's neighbours in CSR order, step j using word 2
 * (cached class) or word 3 (uncached class) of counter (j, v, h-1).  Each
 * row lists its cached picks (Floyd order), then the uncached ones.
 * deg(v) <= k takes the whole row as gnnav_sample does.  Frontier union,
 * blocks and sizes are exactly as gnnav_sample.  async != 0: no final
 * synchronisation (as gnnav_sample_async).  With an updating (FIFO or LRU)
 * cache the slot map is read after the cache's last update (ordered by its
 * event).
 * Errors: as gnnav_sample; E_INVALID also for a NULL cache, a cache of
 * another graph, eta outside [1, 65536], or a fanout above 64.          */
gnnav_status gnnav_sample_biased(const gnnav_graph *g, const gnnav_cache *cache, uint32_t eta,
                                 const int32_t *seeds_dev, int64_t n_seeds, const int32_t *fanouts,
                                 int32_t n_hops, uint64_t rng_seed, gnnav_blocks *blocks,
                                 int32_t async, void *stream);

/* ------------------------------------------------------------ profiling ---
 * Per-kernel timing with HIP events recorded around every kernel launch on
 * the stream it is launched on.  profile_start clears the table and turns
 * recording on; profile_stop synchronises the device, resolves the events
 * and turns recording off.  Entries are read by index.  Both launch an
 * empty kernel, k_profile_mark(1) and k_profile_mark(2), so the recorded
 * region can be found in an external kernel trace.                        */
gnnav_status gnnav_profile_start(void);
gnnav_status gnnav_profile_stop(void);
int32_t gnnav_profile_count(void);
gnnav_status gnnav_profile_get(int32_t i, char *name, int32_t name_cap, int64_t *launches,
                               double *total_ms);

/* Per-launch durations (ms, launch order) of recorded kernel i after
 * gnnav_profile_stop: copies min(cap, count) of them to ms and the count
 * to *n (n may be NULL).  Errors: E_INVALID (i out of range, ms NULL with
 * cap > 0).                                                                */
gnnav_status gnnav_profile_samples(int32_t i, float *ms, int64_t cap, int64_t *n);

/* -------------------------------------------------------------- testing ---
 * Hooks that force failure paths from the host, so tests can reach them
 * while every kernel still runs to its normal end.  Process-wide settings,
 * not meant for production use.
 *
 * gnnav_debug_set_spin_limit: look-back polls after which a device-wide
 * scan's wait gives up (default 2^20).  0 makes every tile after a scan's
 * first give up before its first poll: the scan's results are wrong, every
 * kernel still ends, and the next synchronisation point returns E_DEVICE.
 *
 * gnnav_debug_fail_allocations: after `after` more successful device or
 * pinned host allocations by the library, every further one fails as if
 * memory were exhausted (E_NOMEM); a negative value turns this off.
 * Both always return GNNAV_OK.                                             */
gnnav_status gnnav_debug_set_spin_limit(uint32_t polls);
gnnav_status gnnav_debug_fail_allocations(int64_t after);

#ifdef __cplusplus
}
#endif

#endif /* GNNAV_H */
