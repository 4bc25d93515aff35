/*
 * oracle_checks.c -- drives every entry point of the CPU oracle (oracle/oracle.c)
 * and of the seeded input generator (synth/synth.c) over small and degenerate
 * shapes, for a build with AddressSanitizer and UndefinedBehaviorSanitizer.
 *
 * Test infrastructure: it checks return codes and cheap invariants (indices in
 * range, distances non-negative, the two-best order); the values themselves are
 * pinned by the Python oracle tests. Any out-of-bounds access, use after free,
 * signed overflow, misaligned access or bad shift aborts the run with a report.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/som_oracle.h"
#include "../../synth/synth.h"

static int failures = 0;

#define CHECK(cond)                                                          \
    do {                                                                     \
        if (!(cond)) {                                                       \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                      \
        }                                                                    \
    } while (0)

static void *xmalloc(size_t n) { return malloc(n ? n : 1); }

/* One batch: generate, then run every oracle entry point over the whole map and over a
 * sub-block with a row stride larger than its width. */
static void batch(uint64_t seed, int64_t N, int64_t V, int64_t E, int kind, int nthreads)
{
    const int64_t M = E * E;
    int32_t *rp = xmalloc((size_t)(N + 1) * sizeof *rp);
    const int64_t nnz = synth_csr_row_ptr(seed, N, V, 11.0, rp, nthreads);
    CHECK(nnz >= 0);
    if (nnz < 0) { free(rp); return; }
    int32_t *ci = xmalloc((size_t)nnz * sizeof *ci);
    CHECK(synth_csr_col_idx(seed, N, V, 11.0, 1.1, rp, ci, nthreads) == 0);
    float *vals = xmalloc((size_t)nnz * sizeof *vals);
    CHECK(synth_values(seed, SYNTH_VAL_QUANTISED, nnz, vals, nthreads) == 0);
    CHECK(synth_values(seed, SYNTH_VAL_UNIFORM, nnz, vals, nthreads) == 0);

    float *W = xmalloc((size_t)(V * M) * sizeof *W);
    CHECK(synth_codebook(seed, kind, V, M, 0, V, 0, M, W, M, nthreads) == 0);
    /* a sub-block written into a wider buffer: rows [1, V), neurons [M/3, M) */
    if (V > 1 && M > 2) {
        float *blk = xmalloc((size_t)((V - 1) * (M + 5)) * sizeof *blk);
        CHECK(synth_codebook(seed, kind, V, M, 1, V, M / 3, M, blk, M + 5, nthreads) == 0);
        free(blk);
    }

    int64_t groups = (N + 7) / 8;
    int32_t *td = xmalloc((size_t)groups * sizeof *td);
    CHECK(synth_tile_distinct(rp, ci, N, 8, td, nthreads) == 0);
    for (int64_t t = 0; t < groups; ++t) CHECK(td[t] >= 0 && td[t] <= V);
    free(td);

    int32_t *b1 = xmalloc((size_t)N * sizeof *b1), *b2 = xmalloc((size_t)N * sizeof *b2);
    double *d1 = xmalloc((size_t)N * sizeof *d1), *d2 = xmalloc((size_t)N * sizeof *d2);
    double *d3 = xmalloc((size_t)N * sizeof *d3);
    double *nrm = xmalloc((size_t)M * sizeof *nrm);

    CHECK(som_norms_oracle_host(W, M, V, 0, M, nrm) == SOM_ORACLE_OK);
    CHECK(som_bmu_oracle_host(W, M, V, 0, M, rp, ci, N, b1, d1, d2) == SOM_ORACLE_OK);
    for (int64_t s = 0; s < N; ++s) CHECK(b1[s] >= 0 && b1[s] < M && d1[s] >= 0 && d2[s] >= d1[s]);
    CHECK(som_bmu2_oracle_host(W, M, V, 0, M, rp, ci, N, b1, d1, b2, d2, d3) == SOM_ORACLE_OK);
    for (int64_t s = 0; s < N; ++s) {
        CHECK(b1[s] >= 0 && b1[s] < M && d1[s] >= 0 && d2[s] >= d1[s] && d3[s] >= d2[s]);
        CHECK(M == 1 ? (b2[s] == -1 && isinf(d2[s])) : (b2[s] >= 0 && b2[s] < M && b2[s] != b1[s]));
    }
    CHECK(som_bmu_sf_oracle_host(W, M, V, 0, M, rp, ci, vals, N, b1, d1, b2, d2, d3) == SOM_ORACLE_OK);
    if (M > 2) {
        /* neurons [1, M): a block whose row stride exceeds its width */
        CHECK(som_bmu_oracle_host(W + 1, M, V, 1, M, rp, ci, N, b1, d1, NULL) == SOM_ORACLE_OK);
        for (int64_t s = 0; s < N; ++s) CHECK(b1[s] >= 1 && b1[s] < M);
        CHECK(som_bmu2_oracle_host(W + 1, M, V, 1, M, rp, ci, N, b1, d1, b2, d2, d3) == SOM_ORACLE_OK);
        CHECK(som_norms_oracle_host(W + 1, M, V, 1, M, nrm) == SOM_ORACLE_OK);
    }

    /* the update on the lattice, with the batch's own best units and a few radii (one past the lattice) */
    if (N > 0) {
        CHECK(som_bmu_oracle_host(W, M, V, 0, M, rp, ci, N, b1, d1, NULL) == SOM_ORACLE_OK);
        float *Wout = xmalloc((size_t)(V * M) * sizeof *Wout);
        const int64_t radii[3] = {1, 2, E + 1};
        for (int r = 0; r < 3; ++r) {
            CHECK(som_update_oracle_host(W, V, E, rp, ci, N, b1, radii[r], Wout) == SOM_ORACLE_OK);
            for (int64_t q = 0; q < V * M; ++q) CHECK(Wout[q] >= 0.0f && Wout[q] <= 1.0f);
        }
        free(Wout);
    }

    free(b1); free(b2); free(d1); free(d2); free(d3); free(nrm);
    free(W); free(vals); free(ci); free(rp);
}

/* Argument and CSR checks: every call here must return an error code, not crash. */
static void bad_arguments(void)
{
    float w[4] = {0.25f, 0.5f, 0.75f, 1.0f};
    int32_t rp[3] = {0, 2, 3};
    int32_t ci[3] = {0, 1, 1};
    int32_t b[2];
    double d[2], d2[2], d3[2], n[2];
    int32_t b2[2];
    CHECK(som_bmu_oracle_host(NULL, 2, 2, 0, 2, rp, ci, 2, b, d, d2) == SOM_ORACLE_BAD_ARG);
    CHECK(som_bmu_oracle_host(w, 1, 2, 0, 2, rp, ci, 2, b, d, d2) == SOM_ORACLE_BAD_ARG);  /* ldw < width */
    CHECK(som_bmu_oracle_host(w, 2, 0, 0, 2, rp, ci, 2, b, d, d2) == SOM_ORACLE_BAD_ARG);  /* V < 1 */
    CHECK(som_bmu_oracle_host(w, 2, 2, 1, 1, rp, ci, 2, b, d, d2) == SOM_ORACLE_BAD_ARG);  /* empty block */
    CHECK(som_bmu_oracle_host(w, 2, 2, 0, 2, rp, ci, -1, b, d, d2) == SOM_ORACLE_BAD_ARG);
    CHECK(som_bmu_oracle_host(w, 2, 2, 0, 2, rp, ci, 0, NULL, NULL, NULL) == SOM_ORACLE_OK);  /* N = 0 */
    int32_t bad_rp[3] = {0, 2, 1};
    CHECK(som_bmu_oracle_host(w, 2, 2, 0, 2, bad_rp, ci, 2, b, d, d2) == SOM_ORACLE_BAD_CSR);
    int32_t neg_rp[3] = {-1, 1, 2};  /* offsets before the start of col_idx */
    CHECK(som_bmu_oracle_host(w, 2, 2, 0, 2, neg_rp, ci, 2, b, d, d2) == SOM_ORACLE_BAD_CSR);
    CHECK(som_bmu2_oracle_host(w, 2, 2, 0, 2, neg_rp, ci, 2, b, d, b2, d2, d3) == SOM_ORACLE_BAD_CSR);
    int32_t bad_ci[3] = {0, 5, 1};
    CHECK(som_bmu_oracle_host(w, 2, 2, 0, 2, rp, bad_ci, 2, b, d, d2) == SOM_ORACLE_BAD_CSR);
    int32_t neg_ci[3] = {-1, 0, 1};
    CHECK(som_bmu2_oracle_host(w, 2, 2, 0, 2, rp, neg_ci, 2, b, d, b2, d2, d3) == SOM_ORACLE_BAD_CSR);
    CHECK(som_bmu_sf_oracle_host(w, 2, 2, 0, 2, rp, ci, NULL, 2, b, d, b2, d2, d3) == SOM_ORACLE_BAD_ARG);
    CHECK(som_norms_oracle_host(w, 2, 2, 0, 2, NULL) == SOM_ORACLE_BAD_ARG);
    CHECK(som_norms_oracle_host(w, 2, 2, 0, 2, n) == SOM_ORACLE_OK);
    float out[4];
    CHECK(som_update_oracle_host(w, 1, 2, rp, ci, 2, b, 0, out) == SOM_ORACLE_BAD_ARG);  /* radius 0 */
    int32_t far_bmu[2] = {7, -3};  /* units off the lattice */
    int32_t on_bmu[2] = {3, 0};
    int32_t rp1[3] = {0, 1, 1};
    int32_t ci1[1] = {0};
    CHECK(som_update_oracle_host(w, 1, 2, rp1, ci1, 2, far_bmu, 1, out) == SOM_ORACLE_BAD_ARG);
    CHECK(som_update_oracle_host(w, 1, 2, rp1, ci1, 2, on_bmu, 1, out) == SOM_ORACLE_OK);
    CHECK(synth_codebook(1, 9, 2, 4, 0, 2, 0, 4, out, 4, 1) < 0);          /* unknown kind */
    CHECK(synth_codebook(1, SYNTH_CB_UNIFORM_BLUR3, 1, 3, 0, 1, 0, 3, out, 3, 1) < 0);  /* M not square */
    CHECK(synth_codebook(1, SYNTH_CB_UNIFORM, 1, 4, 0, 1, 2, 1, out, 4, 1) < 0);        /* i1 < i0 */
    CHECK(synth_csr_row_ptr(1, -1, 10, 11.0, rp, 1) < 0);
    CHECK(synth_values(1, 7, 3, out, 1) < 0);
    CHECK(synth_tile_distinct(rp, ci, 2, 0, b, 1) < 0);
}

int main(void)
{
    bad_arguments();
    /* (seed, N, V, E, kind, threads): degenerate, ragged and multi-threaded shapes */
    batch(1, 0, 10, 2, SYNTH_CB_UNIFORM, 1);
    batch(2, 1, 1, 1, SYNTH_CB_QUANTISED, 1);
    batch(3, 17, 5, 3, SYNTH_CB_UNIFORM, 1);     /* rows capped at V = 5 ids */
    batch(4, 40, 300, 4, SYNTH_CB_UNIFORM_BLUR3, 3);
    batch(5, 133, 2000, 5, SYNTH_CB_QUANTISED, 4);
    batch(6, 64, 30000, 3, SYNTH_CB_UNIFORM_BLUR3, 8);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle and synth checks passed\n");
    return 0;
}
