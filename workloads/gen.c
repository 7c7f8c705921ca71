/* Synthetic edge-list generators (input tooling, not part of the method).
 *
 * Chung-Lu and R-MAT pair generators with deduplication and top-up, written
 * in C because the graphs reach 10^8 edges.  Random numbers come from
 * xoshiro256** seeded through splitmix64 (Blackman & Vigna, "Scrambled
 * linear pseudorandom number generators", 2018).  Output: distinct
 * undirected pairs (src[i], dst[i]), src != dst, each pair listed once, node
 * ids passed through a seeded random permutation.
 *
 * Build: gcc -O2 -fPIC -shared -o libgen.so gen.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct { uint64_t s[4]; } rng_t;

static uint64_t splitmix64(uint64_t *x) {
    uint64_t z = (*x += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}
static void rng_init(rng_t *r, uint64_t seed) {
    uint64_t x = seed;
    for (int i = 0; i < 4; ++i) r->s[i] = splitmix64(&x);
}
static inline uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }
static inline uint64_t next64(rng_t *r) {
    uint64_t *s = r->s;
    uint64_t res = rotl(s[1] * 5, 7) * 9, t = s[1] << 17;
    s[2] ^= s[0]; s[3] ^= s[1]; s[1] ^= s[2]; s[0] ^= s[3];
    s[2] ^= t; s[3] = rotl(s[3], 45);
    return res;
}
static inline double unif(rng_t *r) { return (double)(next64(r) >> 11) * 0x1.0p-53; }
static inline uint64_t below(rng_t *r, uint64_t n) { /* n < 2^32 */
    return ((next64(r) >> 32) * n) >> 32;
}

/* LSD radix sort of 64-bit keys in 8-bit digits (digits that are equal
 * across all keys are skipped), then in-place unique. */
static int64_t sort_unique(uint64_t *a, int64_t m, int key_bits) {
    if (m <= 1) return m;
    uint64_t *tmp = (uint64_t *)malloc((size_t)m * sizeof(uint64_t));
    if (!tmp) return -1;
    uint64_t *src = a, *dst = tmp;
    int64_t cnt[256];
    for (int shift = 0; shift < key_bits; shift += 8) {
        memset(cnt, 0, sizeof(cnt));
        for (int64_t i = 0; i < m; ++i) cnt[(src[i] >> shift) & 0xff]++;
        int trivial = 0;
        for (int b = 0; b < 256; ++b) if (cnt[b] == m) trivial = 1;
        if (trivial) continue;
        int64_t run = 0;
        for (int b = 0; b < 256; ++b) { int64_t c = cnt[b]; cnt[b] = run; run += c; }
        for (int64_t i = 0; i < m; ++i) dst[cnt[(src[i] >> shift) & 0xff]++] = src[i];
        uint64_t *t = src; src = dst; dst = t;
    }
    if (src != a) memcpy(a, src, (size_t)m * sizeof(uint64_t));
    free(tmp);
    int64_t u = 1;
    for (int64_t i = 1; i < m; ++i) if (a[i] != a[u - 1]) a[u++] = a[i];
    return u;
}

/* Merge sorted-unique a[0:na] and b[0:nb] into out (sorted, unique). */
static int64_t merge_unique(const uint64_t *a, int64_t na, const uint64_t *b, int64_t nb,
                            uint64_t *out) {
    int64_t i = 0, j = 0, k = 0;
    while (i < na || j < nb) {
        uint64_t x;
        if (j >= nb || (i < na && a[i] <= b[j])) x = a[i++]; else x = b[j++];
        if (k == 0 || out[k - 1] != x) out[k++] = x;
    }
    return k;
}

typedef void (*draw_fn)(void *ctx, rng_t *r, int64_t *u, int64_t *v);

/* Draw pairs until `target` distinct undirected pairs exist; keep exactly
 * `target` of them (a uniform random subset when over); permute ids. */
static int64_t pairs_topped_up(int64_t n, int64_t target, uint64_t seed, draw_fn draw,
                               void *ctx, int32_t *src, int32_t *dst) {
    if (target <= 0) return 0;
    rng_t r; rng_init(&r, seed);
    int key_bits = 8;
    while (key_bits < 64 && ((uint64_t)1 << key_bits) <= (uint64_t)n * (uint64_t)n) key_bits += 8;
    uint64_t *keys = NULL;
    int64_t have = 0;
    for (int round = 0; round < 200 && have < target; ++round) {
        int64_t need = target - have;
        int64_t want = round == 0 ? target + target / 8 + 16 : need * 2 + 16;
        uint64_t *fresh = (uint64_t *)malloc((size_t)want * sizeof(uint64_t));
        if (!fresh) { free(keys); return -1; }
        int64_t m = 0;
        for (int64_t i = 0; i < want; ++i) {
            int64_t u, v;
            draw(ctx, &r, &u, &v);
            if (u < 0 || u == v) continue;
            int64_t lo = u < v ? u : v, hi = u < v ? v : u;
            fresh[m++] = (uint64_t)lo * (uint64_t)n + (uint64_t)hi;
        }
        m = sort_unique(fresh, m, key_bits);
        if (m < 0) { free(fresh); free(keys); return -1; }
        if (!keys) { keys = fresh; have = m; continue; }
        uint64_t *merged = (uint64_t *)malloc((size_t)(have + m) * sizeof(uint64_t));
        if (!merged) { free(fresh); free(keys); return -1; }
        have = merge_unique(keys, have, fresh, m, merged);
        free(keys); free(fresh);
        keys = merged;
    }
    if (have < target) { free(keys); return -2; }
    if (have > target) { /* uniform subset: partial Fisher-Yates, then re-sort */
        for (int64_t i = 0; i < target; ++i) {
            int64_t j = i + (int64_t)below(&r, (uint64_t)(have - i));
            uint64_t t = keys[i]; keys[i] = keys[j]; keys[j] = t;
        }
        sort_unique(keys, target, key_bits);
    }
    int32_t *perm = (int32_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!perm) { free(keys); return -1; }
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
    for (int64_t i = n - 1; i > 0; --i) {
        int64_t j = (int64_t)below(&r, (uint64_t)(i + 1));
        int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
    }
    for (int64_t i = 0; i < target; ++i) {
        src[i] = perm[keys[i] / (uint64_t)n];
        dst[i] = perm[keys[i] % (uint64_t)n];
    }
    free(perm); free(keys);
    return target;
}

/* ---- Chung-Lu: endpoints i.i.d. proportional to capped weights (alias). */
typedef struct { int64_t n; double *prob; int64_t *alias; } cl_ctx;

static void cl_draw1(cl_ctx *c, rng_t *r, int64_t *x) {
    int64_t i = (int64_t)below(r, (uint64_t)c->n);
    *x = unif(r) < c->prob[i] ? i : c->alias[i];
}
static void cl_draw(void *ctx, rng_t *r, int64_t *u, int64_t *v) {
    cl_draw1((cl_ctx *)ctx, r, u);
    cl_draw1((cl_ctx *)ctx, r, v);
}

/* weights w_i ~ (i+1)^(-1/(gamma-1)), capped at sqrt(n*avg), sum n*avg */
int64_t gen_chung_lu_weights(int64_t n, double avg_deg, double gamma, double *w) {
    double total = (double)n * avg_deg, cap = sqrt(total);
    for (int64_t i = 0; i < n; ++i) w[i] = pow((double)(i + 1), -1.0 / (gamma - 1.0));
    for (int it = 0; it < 200; ++it) {
        double s = 0, mx = 0;
        for (int64_t i = 0; i < n; ++i) s += w[i];
        for (int64_t i = 0; i < n; ++i) { w[i] *= total / s; if (w[i] > mx) mx = w[i]; }
        if (mx <= cap * (1 + 1e-12)) break;
        for (int64_t i = 0; i < n; ++i) if (w[i] > cap) w[i] = cap;
    }
    return 0;
}

int64_t gen_chung_lu(int64_t n, double avg_deg, double gamma, uint64_t seed,
                     int32_t *src, int32_t *dst, int64_t target) {
    double *w = (double *)malloc((size_t)n * sizeof(double));
    double *prob = (double *)malloc((size_t)n * sizeof(double));
    int64_t *alias = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    int64_t *small = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    int64_t *large = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    if (!w || !prob || !alias || !small || !large) return -1;
    gen_chung_lu_weights(n, avg_deg, gamma, w);
    /* Vose's alias method */
    double s = 0;
    for (int64_t i = 0; i < n; ++i) s += w[i];
    int64_t ns = 0, nl = 0;
    for (int64_t i = 0; i < n; ++i) {
        prob[i] = w[i] * (double)n / s;
        alias[i] = i;
        if (prob[i] < 1.0) small[ns++] = i; else large[nl++] = i;
    }
    while (ns > 0 && nl > 0) {
        int64_t l = small[--ns], g = large[--nl];
        alias[l] = g;
        prob[g] = (prob[g] + prob[l]) - 1.0;
        if (prob[g] < 1.0) small[ns++] = g; else large[nl++] = g;
    }
    while (nl > 0) prob[large[--nl]] = 1.0;
    while (ns > 0) prob[small[--ns]] = 1.0;
    cl_ctx c = {n, prob, alias};
    int64_t got = pairs_topped_up(n, target, seed, cl_draw, &c, src, dst);
    free(w); free(prob); free(alias); free(small); free(large);
    return got;
}

/* ---- R-MAT: recursive quadrant choice; endpoints >= n rejected. */
typedef struct { int scale; int64_t n; uint32_t a, ab, abc; } rm_ctx;

static void rm_draw(void *ctx, rng_t *r, int64_t *u, int64_t *v) {
    rm_ctx *c = (rm_ctx *)ctx;
    int64_t x = 0, y = 0;
    uint64_t bits = 0;
    for (int l = 0; l < c->scale; ++l) {
        if ((l & 3) == 0) bits = next64(r);
        uint32_t q = (uint32_t)(bits & 0xffff);   /* level draw, 16-bit resolution */
        bits >>= 16;
        int bu = q >= c->ab, bv = (q >= c->a && q < c->ab) || q >= c->abc;
        x = (x << 1) | bu;
        y = (y << 1) | bv;
    }
    if (x >= c->n || y >= c->n) { *u = -1; *v = -1; return; }
    *u = x; *v = y;
}

int64_t gen_rmat(int32_t scale, int64_t n, double a, double b, double c, double d,
                 uint64_t seed, int32_t *src, int32_t *dst, int64_t target) {
    double s = a + b + c + d;
    rm_ctx ctx = {scale, n, (uint32_t)(a / s * 65536.0 + 0.5), (uint32_t)((a + b) / s * 65536.0 + 0.5),
                  (uint32_t)((a + b + c) / s * 65536.0 + 0.5)};
    return pairs_topped_up(n, target, seed, rm_draw, &ctx, src, dst);
}
