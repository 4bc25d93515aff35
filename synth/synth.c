/*
 * synth.c -- seeded synthetic workloads for the sparse-binary BMU search.
 *
 * Test and benchmark infrastructure. It draws inputs (sparse-binary CSR
 * batches and feature-major codebooks) and computes one workload statistic
 * (distinct features per tile of consecutive rows, the unit of the
 * algorithmic-traffic count). It computes no part of the BMU search itself:
 * no distances, no norms, no dot products, no argmin.
 *
 * The inputs stand in for the paper's MEDLINE/MeSH corpus (corpus section,
 * Table 1: sorted descriptor ids per article, binary values implicit), which
 * is not available here. Shapes follow that corpus: about 30k features, a
 * mean of 11-12 active features per row, heavy-tailed feature frequency.
 *
 * Every value is a pure function of (seed, position), built on SplitMix64
 * (Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014): a 64-bit state advanced by the golden-ratio increment, each
 * output passed through the variant-13 64-bit finaliser. Any row of a CSR
 * batch and any block of a codebook can therefore be regenerated on its own,
 * and the result does not depend on the thread count.
 */
#include "synth.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Stream bases: one per kind of draw, so codebook values and CSR draws made
 * from the same seed are unrelated. */
static inline uint64_t csr_base(uint64_t seed) { return mix64(seed ^ 0xA0761D6478BD642FULL); }
static inline uint64_t cb_base(uint64_t seed) { return mix64(seed ^ 0xE7037ED1A0B428DBULL); }
static inline uint64_t val_base(uint64_t seed) { return mix64(seed ^ 0x8EBC6AF09C88C6E3ULL); }

/* ------------------------------------------------------------------ threads */

typedef void (*range_fn)(int64_t begin, int64_t end, void *ctx);

typedef struct {
    range_fn fn;
    void *ctx;
    int64_t begin, end;
} job_t;

static void *run_job(void *p)
{
    job_t *j = (job_t *)p;
    if (j->begin < j->end) j->fn(j->begin, j->end, j->ctx);
    return NULL;
}

/* Split [0, n) into nthreads contiguous chunks (boundaries rounded to
 * multiples of `grain`) and run fn on each. */
static void parallel_for(int64_t n, int64_t grain, int nthreads, range_fn fn, void *ctx)
{
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    if (grain < 1) grain = 1;
    if (nthreads == 1 || n <= grain) {
        if (n > 0) fn(0, n, ctx);
        return;
    }
    job_t jobs[256];
    pthread_t th[256];
    int64_t chunk = (n + nthreads - 1) / nthreads;
    chunk = ((chunk + grain - 1) / grain) * grain;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].fn = fn;
        jobs[t].ctx = ctx;
        jobs[t].begin = (int64_t)t * chunk < n ? (int64_t)t * chunk : n;
        jobs[t].end = (int64_t)(t + 1) * chunk < n ? (int64_t)(t + 1) * chunk : n;
    }
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, run_job, &jobs[t]) != 0) {
            run_job(&jobs[t]); /* no thread: run the chunk here */
            th[t] = 0;
        }
    }
    run_job(&jobs[0]);
    for (int t = 1; t < nthreads; ++t)
        if (th[t]) pthread_join(th[t], NULL);
}

/* --------------------------------------------------------------- codebook */

/* Raw 64-bit draw for feature-major element idx = v*M + i. */
static inline uint64_t cb_draw(uint64_t base, uint64_t idx) { return mix64(base + (idx + 1) * GOLDEN); }

/* U[0,1) with 24 random bits: every value is a multiple of 2^-24, exact in fp32. */
static inline float cb_uniform(uint64_t base, uint64_t idx)
{
    return (float)(cb_draw(base, idx) >> 40) * (1.0f / 16777216.0f);
}

/* k/256 with k uniform on {0..255}. */
static inline float cb_quantised(uint64_t base, uint64_t idx)
{
    return (float)(cb_draw(base, idx) >> 56) * (1.0f / 256.0f);
}

typedef struct {
    uint64_t base;
    int kind;
    int64_t V, M, E;
    int64_t v0, i0, i1;
    float *out;
    int64_t ld;
} cb_ctx;

static void cb_rows(int64_t rb, int64_t re, void *p)
{
    const cb_ctx *c = (const cb_ctx *)p;
    for (int64_t r = rb; r < re; ++r) {
        const int64_t v = c->v0 + r;
        float *dst = c->out + r * c->ld;
        const uint64_t row0 = (uint64_t)v * (uint64_t)c->M;
        if (c->kind == SYNTH_CB_UNIFORM) {
            for (int64_t i = c->i0; i < c->i1; ++i) dst[i - c->i0] = cb_uniform(c->base, row0 + (uint64_t)i);
        } else if (c->kind == SYNTH_CB_QUANTISED) {
            for (int64_t i = c->i0; i < c->i1; ++i) dst[i - c->i0] = cb_quantised(c->base, row0 + (uint64_t)i);
        } else {
            /* 3x3 box mean over the in-bounds lattice neighbours of neuron
             * i = r*E + c, in row-major window order. The summands are
             * multiples of 2^-24 below 1, so the fp64 sum of at most nine is
             * exact; the quotient is rounded once to fp64 and once to fp32. */
            const int64_t E = c->E;
            for (int64_t i = c->i0; i < c->i1; ++i) {
                const int64_t rr = i / E, cc = i % E;
                double sum = 0.0;
                int cnt = 0;
                for (int64_t dr = -1; dr <= 1; ++dr) {
                    const int64_t r2 = rr + dr;
                    if (r2 < 0 || r2 >= E) continue;
                    for (int64_t dc = -1; dc <= 1; ++dc) {
                        const int64_t c2 = cc + dc;
                        if (c2 < 0 || c2 >= E) continue;
                        sum += (double)cb_uniform(c->base, row0 + (uint64_t)(r2 * E + c2));
                        ++cnt;
                    }
                }
                dst[i - c->i0] = (float)(sum / (double)cnt);
            }
        }
    }
}

int synth_codebook(uint64_t seed, int kind, int64_t V, int64_t M, int64_t v0, int64_t v1, int64_t i0,
                   int64_t i1, float *out, int64_t ld, int nthreads)
{
    if (!out || V < 1 || M < 1 || v0 < 0 || v1 > V || v0 > v1 || i0 < 0 || i1 > M || i0 > i1 || ld < i1 - i0)
        return -1;
    int64_t E = 0;
    if (kind == SYNTH_CB_UNIFORM_BLUR3) {
        E = (int64_t)llround(sqrt((double)M));
        while (E * E > M) --E;
        while ((E + 1) * (E + 1) <= M) ++E;
        if (E * E != M) return -2; /* the lattice must be square */
    } else if (kind != SYNTH_CB_UNIFORM && kind != SYNTH_CB_QUANTISED) {
        return -3;
    }
    cb_ctx c = {cb_base(seed), kind, V, M, E, v0, i0, i1, out, ld};
    parallel_for(v1 - v0, 1, nthreads, cb_rows, &c);
    return 0;
}

/* -------------------------------------------------------------------- CSR */

/* Per-row stream: a SplitMix64 generator whose start state is a hash of
 * (seed, row). Draw 0 sets the row's length, later draws its feature ids. */
typedef struct {
    uint64_t state;
} rowrng;

static inline rowrng row_stream(uint64_t base, int64_t row)
{
    rowrng g;
    g.state = mix64(base + ((uint64_t)row + 1) * GOLDEN);
    return g;
}

static inline double next_u53(rowrng *g)
{
    g->state += GOLDEN;
    return (double)(mix64(g->state) >> 11) * (1.0 / 9007199254740992.0);
}

#define POIS_TAB 256

typedef struct {
    double pois_cdf[POIS_TAB]; /* P(K <= k) for K ~ Poisson(lam) */
    int pois_len;
    double *zipf_cdf;          /* P(rank <= k+1), k = 0..V-1 */
    int64_t V;
    uint64_t base;
} csr_tables;

static void build_pois(csr_tables *t, double lam)
{
    double p = exp(-lam), c = p;
    int k = 0;
    t->pois_cdf[0] = c;
    for (k = 1; k < POIS_TAB - 1; ++k) {
        p *= lam / (double)k;
        c += p;
        t->pois_cdf[k] = c;
        if (p < 1e-300 || (k > lam && 1.0 - c < 1e-17)) break;
    }
    t->pois_len = k + 1;
    t->pois_cdf[k] = 1.0;
}

static int build_zipf(csr_tables *t, int64_t V, double s)
{
    t->zipf_cdf = (double *)malloc((size_t)V * sizeof(double));
    if (!t->zipf_cdf) return -1;
    double acc = 0.0;
    for (int64_t k = 0; k < V; ++k) {
        acc += pow((double)(k + 1), -s);
        t->zipf_cdf[k] = acc;
    }
    for (int64_t k = 0; k < V; ++k) t->zipf_cdf[k] /= acc;
    t->zipf_cdf[V - 1] = 1.0;
    t->V = V;
    return 0;
}

/* first index j with u < cdf[j] (u < 1 = cdf[n-1], so j exists) */
static inline int64_t first_above(const double *cdf, int64_t n, double u)
{
    int64_t lo = 0, hi = n - 1;
    while (lo < hi) {
        int64_t mid = lo + ((hi - lo) >> 1);
        if (u < cdf[mid]) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

static inline int64_t row_len(const csr_tables *t, rowrng *g)
{
    const double u = next_u53(g);
    int64_t k = first_above(t->pois_cdf, t->pois_len, u);
    int64_t n = 1 + k;
    return n < t->V ? n : t->V;
}

typedef struct {
    const csr_tables *t;
    int32_t *row_len_out; /* N entries */
} len_ctx;

static void len_rows(int64_t b, int64_t e, void *p)
{
    const len_ctx *c = (const len_ctx *)p;
    for (int64_t s = b; s < e; ++s) {
        rowrng g = row_stream(c->t->base, s);
        c->row_len_out[s] = (int32_t)row_len(c->t, &g);
    }
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

typedef struct {
    const csr_tables *t;
    const int32_t *row_ptr;
    int32_t *col_idx;
} ids_ctx;

static void ids_rows(int64_t b, int64_t e, void *p)
{
    const ids_ctx *c = (const ids_ctx *)p;
    const int64_t V = c->t->V;
    for (int64_t s = b; s < e; ++s) {
        rowrng g = row_stream(c->t->base, s);
        const int64_t n = row_len(c->t, &g);
        int32_t *ids = c->col_idx + c->row_ptr[s];
        int64_t have = 0;
        int64_t tries = 0;
        /* Zipf draws without replacement: a repeat is rejected and drawn
         * again, which gives the distribution of successive sampling without
         * replacement. After 1000*n rejections (only reachable when n is
         * close to V) the remaining slots take the lowest unused ids. */
        while (have < n && tries < 1000 * n + 1000) {
            const int32_t id = (int32_t)first_above(c->t->zipf_cdf, V, next_u53(&g));
            ++tries;
            int dup = 0;
            for (int64_t j = 0; j < have; ++j)
                if (ids[j] == id) { dup = 1; break; }
            if (!dup) ids[have++] = id;
        }
        for (int32_t id = 0; have < n; ++id) {
            int dup = 0;
            for (int64_t j = 0; j < have; ++j)
                if (ids[j] == id) { dup = 1; break; }
            if (!dup) ids[have++] = id;
        }
        if (n <= 64) { /* insertion sort: rows are short */
            for (int64_t j = 1; j < n; ++j) {
                int32_t x = ids[j];
                int64_t k = j - 1;
                while (k >= 0 && ids[k] > x) { ids[k + 1] = ids[k]; --k; }
                ids[k + 1] = x;
            }
        } else {
            qsort(ids, (size_t)n, sizeof(int32_t), cmp_i32);
        }
    }
}

int64_t synth_csr_row_ptr(uint64_t seed, int64_t N, int64_t V, double lam, int32_t *row_ptr, int nthreads)
{
    if (!row_ptr || N < 0 || V < 1 || !(lam >= 0.0) || lam > 1e4) return -1;
    csr_tables t;
    memset(&t, 0, sizeof t);
    build_pois(&t, lam);
    t.V = V;
    t.base = csr_base(seed);
    /* row lengths land in row_ptr[1..N], then an in-place prefix sum */
    len_ctx c = {&t, row_ptr + 1};
    parallel_for(N, 4096, nthreads, len_rows, &c);
    row_ptr[0] = 0;
    int64_t acc = 0;
    for (int64_t s = 1; s <= N; ++s) {
        acc += row_ptr[s];
        if (acc > 2147483647LL) return -2; /* int32 CSR offsets would overflow */
        row_ptr[s] = (int32_t)acc;
    }
    return acc;
}

int synth_csr_col_idx(uint64_t seed, int64_t N, int64_t V, double lam, double zipf_s, const int32_t *row_ptr,
                      int32_t *col_idx, int nthreads)
{
    if (!row_ptr || (!col_idx && N > 0) || N < 0 || V < 1 || !(lam >= 0.0) || !(zipf_s > 0.0)) return -1;
    csr_tables t;
    memset(&t, 0, sizeof t);
    build_pois(&t, lam);
    if (build_zipf(&t, V, zipf_s) != 0) return -2;
    t.base = csr_base(seed);
    ids_ctx c = {&t, row_ptr, col_idx};
    parallel_for(N, 4096, nthreads, ids_rows, &c);
    free(t.zipf_cdf);
    return 0;
}

/* ---------------------------------------------------- workload statistic */

typedef struct {
    const int32_t *row_ptr, *col_idx;
    int64_t N, TA;
    int32_t *out;
} tile_ctx;

static void tile_rows(int64_t b, int64_t e, void *p)
{
    const tile_ctx *c = (const tile_ctx *)p;
    int32_t *buf = NULL;
    size_t cap = 0;
    for (int64_t t = b; t < e; ++t) {
        const int64_t s0 = t * c->TA;
        const int64_t s1 = s0 + c->TA < c->N ? s0 + c->TA : c->N;
        const int64_t lo = c->row_ptr[s0], hi = c->row_ptr[s1];
        const size_t n = (size_t)(hi - lo);
        if (n > cap) {
            free(buf);
            cap = n * 2;
            buf = (int32_t *)malloc(cap * sizeof(int32_t));
            if (!buf) { c->out[t] = -1; cap = 0; continue; }
        }
        memcpy(buf, c->col_idx + lo, n * sizeof(int32_t));
        qsort(buf, n, sizeof(int32_t), cmp_i32);
        int32_t d = 0;
        for (size_t k = 0; k < n; ++k)
            if (k == 0 || buf[k] != buf[k - 1]) ++d;
        c->out[t] = d;
    }
    free(buf);
}

int synth_tile_distinct(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t TA, int32_t *out,
                        int nthreads)
{
    if (!row_ptr || !out || N < 0 || TA < 1) return -1;
    tile_ctx c = {row_ptr, col_idx, N, TA, out};
    parallel_for((N + TA - 1) / TA, 1024, nthreads, tile_rows, &c);
    return 0;
}

/* ------------------------------------------------------------------ values */

typedef struct {
    uint64_t base;
    int kind;
    float *out;
} val_ctx;

static void val_range(int64_t b, int64_t e, void *p)
{
    const val_ctx *c = (const val_ctx *)p;
    for (int64_t q = b; q < e; ++q) {
        const uint64_t h = mix64(c->base + ((uint64_t)q + 1) * GOLDEN);
        c->out[q] = c->kind == SYNTH_VAL_QUANTISED ? (float)((h >> 56) + 1) * (1.0f / 256.0f)
                                                   : (float)((h >> 40) + 1) * 0x1p-24f;
    }
}

int synth_values(uint64_t seed, int kind, int64_t n, float *out, int nthreads)
{
    if (n < 0 || (n > 0 && !out) || (kind != SYNTH_VAL_UNIFORM && kind != SYNTH_VAL_QUANTISED)) return -1;
    val_ctx c = {val_base(seed), kind, out};
    parallel_for(n, 4096, nthreads, val_range, &c);
    return 0;
}
