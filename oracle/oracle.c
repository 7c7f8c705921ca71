/* Oracle for the sampled mini-batch step of GraphSAGE-style training.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded
 * definition of what the hot path computes.  Only the tests, the smoke check
 * and the bench's CPU-baseline leg may load it.  It shares no code, header,
 * table or helper with the HIP library.
 *
 * What it follows (GNNavigator, DAC'24, arXiv 2404.09544):
 *   - Algorithm 1 (Section 2.1): per mini-batch, sample a subgraph from the
 *     target vertices, bring its data to the device, then per layer
 *     Aggregate and Combine.  Only the forward pass is defined here.
 *   - Eq. 1 (Section 2.1): a_v = Aggregate(h_u | u in N(v), plus h_v);
 *     h_v = Combine(a_v).  Here: GraphSAGE mean aggregation over the sampled
 *     neighbours, combined with the vertex's own row by one linear map.
 *   - Eq. 2 (Section 3.2, "Sampling strategies"): B^l is the union, over the
 *     targets v of B^(l-1), of neighbours selected with probability
 *     k^l / |N(v)|.  Here: min(deg, k) distinct neighbours chosen uniformly
 *     without replacement (each neighbour's inclusion probability is k/deg),
 *     the union taken as an ordered, deduplicated frontier.
 *   - Section 3.2, "Transmission strategies": the device cache finds which
 *     part of the batch is cached; the rest comes from the host store.  With
 *     cache updates disabled and a cache ratio r this is the static
 *     PaGraph-style cache of Section 3.2 ("Reconfigurable runtime backend")
 *     and Section 4.1, filled with the highest-degree vertices.
 *   - Eq. 12 (Section 3.3): |V_i| <= |B^0| * prod_l (1 + k^l), the bound the
 *     frontier sizes obey when tau = 1 and nothing overlaps.
 *
 * Conventions the paper leaves open (the readings are recorded with the
 * design notes): Philox4x32-10 draws keyed by (rng_seed) with counter
 * (slot j, node lo, node hi, hop); range reduction floor(x*b / 2^32);
 * Floyd's subset selection; fanouts[0] applies to the seeds; every node of
 * B^(l-1) is sampled again at hop l; frontiers are ordered "previous
 * frontier, then new ids in first-occurrence order"; seeds are deduplicated
 * keeping first occurrences; cache size floor(r*n) with ties in degree
 * broken by smaller id; the mean over an empty set is the zero vector.
 *
 * Arithmetic for the forward pass is IEEE double.  When the bf16 mode is on,
 * the aggregate and the hidden layers are rounded to bfloat16 (round to
 * nearest, ties to even) exactly where the device path stores bf16.
 *
 * Build: gcc -O2 -fPIC -shared -o liboracle.so oracle.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ O1 ---
 * CSR of an undirected simple graph.  Every input pair (u, v) contributes
 * u->v and, when symmetrize is set, v->u.  Self pairs are dropped and
 * repeated pairs kept once.  Rows list their neighbours in ascending order.
 * row_ptr has n+1 entries; col must hold 2*m entries (the most possible).
 * Returns nnz, or -1 for an endpoint outside [0, n), -2 for no memory.    */
static int cmp_i32(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

int64_t oracle_build_csr(int64_t n, int64_t m, const int32_t *src, const int32_t *dst,
                         int32_t symmetrize, int64_t *row_ptr, int32_t *col) {
    int64_t *fill = (int64_t *)calloc((size_t)(n + 1), sizeof(int64_t));
    if (!fill) return -2;
    for (int64_t i = 0; i < m; ++i) {
        if (src[i] < 0 || src[i] >= n || dst[i] < 0 || dst[i] >= n) { free(fill); return -1; }
    }
    /* count directed arcs per source row (self pairs excluded) */
    for (int64_t i = 0; i <= n; ++i) row_ptr[i] = 0;
    for (int64_t i = 0; i < m; ++i) {
        if (src[i] == dst[i]) continue;
        row_ptr[src[i] + 1]++;
        if (symmetrize) row_ptr[dst[i] + 1]++;
    }
    for (int64_t v = 0; v < n; ++v) row_ptr[v + 1] += row_ptr[v];
    for (int64_t v = 0; v < n; ++v) fill[v] = row_ptr[v];
    for (int64_t i = 0; i < m; ++i) {
        if (src[i] == dst[i]) continue;
        col[fill[src[i]]++] = dst[i];
        if (symmetrize) col[fill[dst[i]]++] = src[i];
    }
    /* sort each row and drop repeats, compacting in place */
    int64_t out = 0;
    for (int64_t v = 0; v < n; ++v) {
        int64_t b = row_ptr[v], e = row_ptr[v + 1];
        qsort(col + b, (size_t)(e - b), sizeof(int32_t), cmp_i32);
        row_ptr[v] = out;
        for (int64_t p = b; p < e; ++p) {
            if (p > b && col[p] == col[p - 1]) continue;
            col[out++] = col[p];
        }
    }
    row_ptr[n] = out;
    free(fill);
    return out;
}

/* ------------------------------------------------------------------ O2 ---
 * Static degree-ranked cache.  rank[] lists all vertices by degree,
 * largest first, equal degrees by smaller id first.  The first
 * C = floor(r * n) of them are cached: slot_map[v] = position of v in
 * rank if that position is < C, else -1.  Returns C.                      */
static const int64_t *g_rank_rowptr;
static int cmp_rank(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    int64_t dx = g_rank_rowptr[x + 1] - g_rank_rowptr[x];
    int64_t dy = g_rank_rowptr[y + 1] - g_rank_rowptr[y];
    if (dx != dy) return dx > dy ? -1 : 1;
    return (x > y) - (x < y);
}

int64_t oracle_rank_cache(int64_t n, const int64_t *row_ptr, double r, int32_t *rank,
                          int32_t *slot_map) {
    for (int64_t v = 0; v < n; ++v) rank[v] = (int32_t)v;
    g_rank_rowptr = row_ptr;
    qsort(rank, (size_t)n, sizeof(int32_t), cmp_rank);
    int64_t c = (int64_t)floor(r * (double)n);
    if (c < 0) c = 0;
    if (c > n) c = n;
    for (int64_t v = 0; v < n; ++v) slot_map[v] = -1;
    for (int64_t s = 0; s < c; ++s) slot_map[rank[s]] = (int32_t)s;
    return c;
}

/* ------------------------------------------------------------------ O3 ---
 * Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw: "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11).  A round multiplies counter words 0
 * and 2 by the two Philox multipliers; the new words are
 * (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0)).
 * Between rounds the key is advanced by the two Weyl constants.           */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    uint32_t k[2] = {key_in[0], key_in[1]};
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k[0] += PHILOX_W0; k[1] += PHILOX_W1; }
        uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
        uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k[0];
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k[1];
        uint32_t n3 = (uint32_t)p0;
        c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
    }
    out[0] = c[0]; out[1] = c[1]; out[2] = c[2]; out[3] = c[3];
}

/* The sampler's draw for (rng_seed, hop, node v, slot j): word 0 of Philox
 * with key (lo32 seed, hi32 seed) and counter (j, lo32 v, hi32 v, hop).    */
uint32_t oracle_draw(uint64_t rng_seed, uint32_t hop, int64_t v, uint32_t j) {
    uint32_t ctr[4] = {j, (uint32_t)((uint64_t)v & 0xffffffffu), (uint32_t)((uint64_t)v >> 32), hop};
    uint32_t key[2] = {(uint32_t)(rng_seed & 0xffffffffu), (uint32_t)(rng_seed >> 32)};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    return out[0];
}

/* ------------------------------------------------------------------ O4 ---
 * A draw x in [0, 2^32) mapped to [0, b): floor(x * b / 2^32).            */
uint32_t oracle_below(uint32_t x, uint32_t b) {
    return (uint32_t)(((uint64_t)x * (uint64_t)b) >> 32);
}

/* ------------------------------------------------------------------ O5 ---
 * Neighbours of v picked at hop `hop` (0-based) with fanout k.
 * deg <= k (or k < 0): the whole row, in CSR order.
 * deg > k: Floyd's algorithm (Bentley & Floyd, "Programming pearls: a
 * sample of brilliance", CACM 1987).  For j = 0..k-1 with m = deg-k+j, draw
 * t uniform in [0, m]; take t unless t was already taken, else take m.  The
 * taken row offsets form a uniform random k-subset.  Output is in j order.
 * Writes global neighbour ids to out and returns how many.               */
int64_t oracle_sample_node(const int64_t *row_ptr, const int32_t *col, int64_t v, int32_t k,
                           uint64_t rng_seed, uint32_t hop, int32_t *out) {
    int64_t start = row_ptr[v];
    int64_t deg = row_ptr[v + 1] - start;
    if (k < 0 || deg <= k) {
        for (int64_t j = 0; j < deg; ++j) out[j] = col[start + j];
        return deg;
    }
    int64_t *taken = (int64_t *)malloc((size_t)(k > 0 ? k : 1) * sizeof(int64_t));
    for (int32_t j = 0; j < k; ++j) {
        int64_t m = deg - k + j;
        int64_t t = oracle_below(oracle_draw(rng_seed, hop, v, (uint32_t)j), (uint32_t)(m + 1));
        int seen = 0;
        for (int32_t i = 0; i < j; ++i)
            if (taken[i] == t) seen = 1;
        taken[j] = seen ? m : t;
        out[j] = col[start + taken[j]];
    }
    free(taken);
    return k;
}

/* ----------------------------------------------------------------- O5b ---
 * Locality-biased neighbour selection: the neighbour-selection probability
 * of Eq. 2 made a function of data locality, p(eta), preferring vertices
 * already in the device cache.  Reading: successive sampling without
 * replacement (k picks, each among the not-yet-picked neighbours with
 * probability proportional to its weight) with weight eta for a cached
 * neighbour (slot_map >= 0) and 1 for an uncached one; eta = 1 is uniform.
 * With two weight classes successive sampling splits into
 *   1. the class of each pick j = 0..k-1, in order: with c_r cached and u_r
 *      uncached neighbours left, t = floor(x * (eta*c_r + u_r) / 2^32) for
 *      x = Philox word 1 of counter (j, v, hop); cached when t < eta*c_r;
 *   2. which members of each class: a uniform subset of the class's size,
 *      by Floyd's algorithm over the class's neighbours in CSR order, with
 *      Philox word 2 (cached class) or word 3 (uncached class) of counter
 *      (j', v, hop) for its j'-th step.
 * Output: the cached picks in Floyd order, then the uncached picks.
 * deg <= k (or k < 0): the whole row, as in O5.                           */
static uint32_t oracle_word(uint64_t rng_seed, uint32_t hop, int64_t v, uint32_t j, int w) {
    uint32_t ctr[4] = {j, (uint32_t)((uint64_t)v & 0xffffffffu), (uint32_t)((uint64_t)v >> 32), hop};
    uint32_t key[2] = {(uint32_t)(rng_seed & 0xffffffffu), (uint32_t)(rng_seed >> 32)};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    return out[w];
}

/* floor(x * b / 2^32) for b up to 2^64 (exact, 128-bit product) */
uint64_t oracle_below64(uint32_t x, uint64_t b) {
    return (uint64_t)(((unsigned __int128)x * (unsigned __int128)b) >> 32);
}

/* Floyd's k-subset of [0, size) with draws from Philox word w; writes the
 * chosen indices in step order. */
static void oracle_floyd(int64_t size, int32_t k, uint64_t rng_seed, uint32_t hop, int64_t v, int w,
                         int64_t *taken) {
    for (int32_t j = 0; j < k; ++j) {
        int64_t m = size - k + j;
        int64_t t = oracle_below(oracle_word(rng_seed, hop, v, (uint32_t)j, w), (uint32_t)(m + 1));
        int seen = 0;
        for (int32_t i = 0; i < j; ++i)
            if (taken[i] == t) seen = 1;
        taken[j] = seen ? m : t;
    }
}

int64_t oracle_sample_node_biased(const int64_t *row_ptr, const int32_t *col, int64_t v, int32_t k,
                                  uint64_t rng_seed, uint32_t hop, const int32_t *slot_map, uint32_t eta,
                                  int32_t *out) {
    int64_t start = row_ptr[v];
    int64_t deg = row_ptr[v + 1] - start;
    if (k < 0 || deg <= k) {
        for (int64_t j = 0; j < deg; ++j) out[j] = col[start + j];
        return deg;
    }
    int64_t *cached = (int64_t *)malloc((size_t)deg * sizeof(int64_t));
    int64_t *uncached = (int64_t *)malloc((size_t)deg * sizeof(int64_t));
    int64_t *taken = (int64_t *)malloc((size_t)(k > 0 ? k : 1) * sizeof(int64_t));
    int64_t c = 0, u = 0;
    for (int64_t i = 0; i < deg; ++i) {
        if (slot_map[col[start + i]] >= 0) cached[c++] = start + i;
        else uncached[u++] = start + i;
    }
    int32_t kc = 0;
    int64_t cr = c, ur = u;
    for (int32_t j = 0; j < k; ++j) {
        uint64_t heavy = (uint64_t)eta * (uint64_t)cr;
        uint64_t t = oracle_below64(oracle_word(rng_seed, hop, v, (uint32_t)j, 1), heavy + (uint64_t)ur);
        if (t < heavy) { kc++; cr--; }
        else ur--;
    }
    int32_t ku = k - kc;
    oracle_floyd(c, kc, rng_seed, hop, v, 2, taken);
    for (int32_t j = 0; j < kc; ++j) out[j] = col[cached[taken[j]]];
    oracle_floyd(u, ku, rng_seed, hop, v, 3, taken);
    for (int32_t j = 0; j < ku; ++j) out[kc + j] = col[uncached[taken[j]]];
    free(cached);
    free(uncached);
    free(taken);
    return k;
}

/* ------------------------------------------------------------------ O6 ---
 * L-hop expansion with relabelling.
 *   F_0 = seeds with repeats removed (first occurrence kept).
 *   For h = 1..L: every node of F_(h-1), in order, is sampled with fanout
 *   fanouts[h-1] and hop counter h-1; N_h is the concatenation of those
 *   samples; F_h = F_(h-1) followed by the ids of N_h not yet present, in
 *   order of first occurrence; indices_h[p] = position of N_h[p] in F_h;
 *   indptr_h is the running count of samples per row of F_(h-1).
 * All frontiers share `nodes` (F_(h-1) is a prefix of F_h); sizes[h] =
 * |F_h|.  Per hop h (1-based), indptr[h-1] holds |F_(h-1)|+1 entries and
 * nbrs[h-1] / indices[h-1] hold E_h entries; caller sizes them to the
 * bounds E_h <= |F_(h-1)| * k_h and |F_h| <= |F_(h-1)| * (1 + k_h).
 * With bias_slot_map != NULL every hop uses the locality-biased selection
 * of O5b with that cache map and eta.
 * Returns 0, or -1 when a seed lies outside [0, n).                      */
int32_t oracle_sample_blocks(int64_t n, const int64_t *row_ptr, const int32_t *col,
                             const int32_t *seeds, int64_t n_seeds, const int32_t *fanouts,
                             int32_t n_hops, uint64_t rng_seed, const int32_t *bias_slot_map, uint32_t eta,
                             int32_t *nodes, int64_t *sizes, int32_t **indptr, int32_t **nbrs,
                             int32_t **indices) {
    int64_t *pos = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    for (int64_t v = 0; v < n; ++v) pos[v] = -1;
    int64_t cnt = 0;
    for (int64_t i = 0; i < n_seeds; ++i) {
        int32_t s = seeds[i];
        if (s < 0 || s >= n) { free(pos); return -1; }
        if (pos[s] < 0) { pos[s] = cnt; nodes[cnt++] = s; }
    }
    sizes[0] = cnt;
    for (int32_t h = 1; h <= n_hops; ++h) {
        int64_t n_prev = cnt, e = 0;
        int32_t *ip = indptr[h - 1], *nb = nbrs[h - 1], *ix = indices[h - 1];
        for (int64_t i = 0; i < n_prev; ++i) {
            ip[i] = (int32_t)e;
            if (bias_slot_map)
                e += oracle_sample_node_biased(row_ptr, col, nodes[i], fanouts[h - 1], rng_seed,
                                               (uint32_t)(h - 1), bias_slot_map, eta, nb + e);
            else
                e += oracle_sample_node(row_ptr, col, nodes[i], fanouts[h - 1], rng_seed,
                                        (uint32_t)(h - 1), nb + e);
        }
        ip[n_prev] = (int32_t)e;
        for (int64_t p = 0; p < e; ++p) {
            int32_t u = nb[p];
            if (pos[u] < 0) { pos[u] = cnt; nodes[cnt++] = u; }
            ix[p] = (int32_t)pos[u];
        }
        sizes[h] = cnt;
    }
    free(pos);
    return 0;
}

/* ------------------------------------------------------------------ O7 ---
 * Feature gather through the cache: out row i = features row ids[i] (a
 * bitwise copy of row_bytes bytes).  A request is a hit when the vertex is
 * cached (slot_map >= 0), a miss otherwise; an id outside [0, n) gives a
 * zero row and counts as invalid.  counts = {hits, misses, invalid}.  When
 * misses is not NULL it receives the missed vertices in request order.   */
void oracle_gather(int64_t n, const uint8_t *features, int64_t row_bytes, const int32_t *slot_map,
                   const int32_t *ids, int64_t n_ids, uint8_t *out, int64_t *counts, int32_t *misses) {
    counts[0] = counts[1] = counts[2] = 0;
    for (int64_t i = 0; i < n_ids; ++i) {
        int32_t v = ids[i];
        if (v < 0 || v >= n) {
            memset(out + i * row_bytes, 0, (size_t)row_bytes);
            counts[2]++;
            continue;
        }
        memcpy(out + i * row_bytes, features + (int64_t)v * row_bytes, (size_t)row_bytes);
        if (slot_map[v] >= 0) {
            counts[0]++;
        } else {
            if (misses) misses[counts[1]] = v;
            counts[1]++;
        }
    }
}

/* ------------------------------------------------------------- O7 (cont.)
 * Cache update after a batch (Section 3.2, "Transmission strategies": the
 * cache is finally updated according to its update policy; its cost is
 * t_replace of Eq. 5).  Policy FIFO over a ring of slots
 * [ring_lo, ring_lo + ring_n): the batch's misses are admitted one by one
 * in request order; each takes the slot under the ring pointer, whose
 * previous vertex (if any) is evicted -- unmapped if the slot map still
 * points at this slot (a vertex requested twice in one batch is admitted
 * twice; it keeps its later slot, and evicting the earlier copy must not
 * unmap it) -- and the pointer advances by one (wrapping).  owner[slot] is
 * the vertex in a slot or -1.                                             */
void oracle_cache_fifo_admit(int32_t *slot_map, int32_t *owner, int64_t ring_lo, int64_t ring_n, int64_t *ptr,
                             const int32_t *misses, int64_t m) {
    for (int64_t i = 0; i < m; ++i) {
        int64_t s = ring_lo + *ptr;
        if (owner[s] >= 0 && slot_map[owner[s]] == (int32_t)s) slot_map[owner[s]] = -1;
        owner[s] = misses[i];
        slot_map[misses[i]] = (int32_t)s;
        *ptr = (*ptr + 1) % ring_n;
    }
}

/* Policy LRU over the same ring of slots.  `order` lists the ring's slots
 * from least to most recently used, as a circular list that starts at
 * order[*head].  Recency is counted in batches: every request of one batch
 * is a use at the same time.  After a gather that hit the slots
 * hit_slots[0..n_hits) (any slots, repeats allowed; those outside the ring
 * are ignored) and missed misses[0..m) (request order):
 *   1. the ring slots hit by the batch become the most recently used, after
 *      every slot it did not touch; each group keeps its earlier relative
 *      order (ties within a batch go to the earlier recency);
 *   2. the misses are admitted one by one in request order, as in FIFO: each
 *      takes the least recently used slot, whose vertex is evicted (unmapped
 *      if the slot map still points at the slot), and that slot becomes the
 *      most recently used.
 * With no ring slot ever hit this is the FIFO policy above.               */
void oracle_cache_lru_update(int32_t *slot_map, int32_t *owner, int64_t ring_lo, int64_t ring_n, int32_t *order,
                             int64_t *head, const int32_t *hit_slots, int64_t n_hits, const int32_t *misses,
                             int64_t m) {
    if (ring_n <= 0) return;
    /* step 1: stable partition of the recency list (untouched, then hit) */
    unsigned char *hit = calloc((size_t)ring_n, 1);
    int32_t *list = malloc((size_t)ring_n * sizeof(int32_t));
    for (int64_t i = 0; i < n_hits; ++i) {
        int64_t s = hit_slots[i];
        if (s >= ring_lo && s < ring_lo + ring_n) hit[s - ring_lo] = 1;
    }
    int64_t k = 0;
    for (int pass = 0; pass < 2; ++pass)
        for (int64_t j = 0; j < ring_n; ++j) {
            int32_t s = order[(*head + j) % ring_n];
            if (hit[s - ring_lo] == pass) list[k++] = s;
        }
    for (int64_t j = 0; j < ring_n; ++j) order[j] = list[j];
    *head = 0;
    /* step 2: admissions, least recently used slot first */
    for (int64_t i = 0; i < m; ++i) {
        int32_t s = order[*head];
        if (owner[s] >= 0 && slot_map[owner[s]] == s) slot_map[owner[s]] = -1;
        owner[s] = misses[i];
        slot_map[misses[i]] = s;
        /* the slot leaves the front and rejoins at the back: in the circular
         * list that is the same cell with the start moved past it */
        *head = (*head + 1) % ring_n;
    }
    free(hit);
    free(list);
}

/* ------------------------------------------------------------- bf16 RNE ---
 * Nearest bfloat16 value of a double, ties to even (IEEE 754-2008 binary
 * rounding with 8 significant bits, exponent range of binary32).  Values at
 * or beyond the overflow threshold become +-inf; NaN stays NaN.  Returned
 * as a double (exactly representable).                                    */
double oracle_round_bf16(double x) {
    if (isnan(x) || isinf(x) || x == 0.0) return x;
    double ax = fabs(x);
    int e;
    frexp(ax, &e);                 /* ax = f * 2^e, f in [0.5, 1) */
    int exp2 = e - 1;              /* 2^exp2 <= ax < 2^(exp2+1) */
    if (exp2 < -126) exp2 = -126;  /* subnormal spacing */
    double ulp = ldexp(1.0, exp2 - 7);
    double q = ax / ulp;           /* exact: power-of-two scaling */
    double fl = floor(q), rem = q - fl, r;
    if (rem > 0.5) r = fl + 1;
    else if (rem < 0.5) r = fl;
    else r = fmod(fl, 2.0) == 0.0 ? fl : fl + 1;
    double y = r * ulp;
    double max_finite = ldexp(255.0, 120); /* (2 - 2^-7) * 2^127 */
    if (y > max_finite) y = INFINITY;
    return x < 0 ? -y : y;
}

void oracle_round_bf16_array(const double *x, double *y, int64_t n) {
    for (int64_t i = 0; i < n; ++i) y[i] = oracle_round_bf16(x[i]);
}

/* ------------------------------------------------------------------ O8 ---
 * One SAGE layer over one block (Eq. 1 with mean aggregation).
 *   agg_i = (1/cnt_i) * sum over p in row i of X[indices[p]], 0 if cnt_i = 0
 *   z_i   = X[i] * W[0:d_in] + agg_i * W[d_in:2*d_in]
 *   out_i = relu(z_i) if relu, else z_i
 * X is n_src x d_in (row stride ld_x), the destination rows are its first
 * n_dst rows.  W is row-major [2*d_in, d_out].  With bf16 set, agg_i is
 * rounded to bfloat16 before the combine, and out_i too when round_out.
 * Only rows listed in `rows` (n_rows of them, or all when rows == NULL) are
 * computed; out row r of the result is destination row rows[r].          */
void oracle_sage_layer(int64_t n_dst, const int32_t *indptr, const int32_t *indices,
                       const double *X, int64_t ld_x, int64_t d_in, const double *W,
                       int64_t d_out, int32_t relu, int32_t bf16, int32_t round_out,
                       const int64_t *rows, int64_t n_rows, double *out, double *agg_out) {
    double *agg = (double *)malloc((size_t)(d_in > 0 ? d_in : 1) * sizeof(double));
    int64_t total = rows ? n_rows : n_dst;
    for (int64_t r = 0; r < total; ++r) {
        int64_t i = rows ? rows[r] : r;
        int64_t b = indptr[i], e = indptr[i + 1];
        for (int64_t c = 0; c < d_in; ++c) agg[c] = 0.0;
        for (int64_t p = b; p < e; ++p) {
            const double *xs = X + (int64_t)indices[p] * ld_x;
            for (int64_t c = 0; c < d_in; ++c) agg[c] += xs[c];
        }
        for (int64_t c = 0; c < d_in; ++c) {
            agg[c] = e > b ? agg[c] / (double)(e - b) : 0.0;
            if (bf16) agg[c] = oracle_round_bf16(agg[c]);
        }
        if (agg_out)
            for (int64_t c = 0; c < d_in; ++c) agg_out[r * d_in + c] = agg[c];
        double *z = out + r * d_out;
        for (int64_t j = 0; j < d_out; ++j) z[j] = 0.0;
        const double *xi = X + i * ld_x;
        for (int64_t c = 0; c < d_in; ++c) {
            const double a = xi[c], *wr = W + c * d_out;
            for (int64_t j = 0; j < d_out; ++j) z[j] += a * wr[j];
        }
        for (int64_t c = 0; c < d_in; ++c) {
            const double a = agg[c], *wr = W + (d_in + c) * d_out;
            for (int64_t j = 0; j < d_out; ++j) z[j] += a * wr[j];
        }
        for (int64_t j = 0; j < d_out; ++j) {
            if (relu && z[j] < 0.0) z[j] = 0.0;
            if (bf16 && round_out) z[j] = oracle_round_bf16(z[j]);
        }
    }
    free(agg);
}
