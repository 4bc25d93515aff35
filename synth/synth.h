/*
 * synth.h -- seeded synthetic workloads for the sparse-binary BMU search.
 *
 * Test and benchmark infrastructure only: it draws inputs and counts a
 * workload statistic, and computes no part of the search. All functions are
 * host-only, thread-safe, and return 0 (or a non-negative count) on success
 * and a negative value on bad arguments. Output buffers belong to the caller.
 */
#ifndef SYNTH_H
#define SYNTH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SYNTH_CB_UNIFORM = 0,       /* U[0,1), 24 random bits per value          */
    SYNTH_CB_QUANTISED = 1,     /* k/256, k uniform on {0..255}              */
    SYNTH_CB_UNIFORM_BLUR3 = 2  /* U[0,1), then the in-bounds 3x3 lattice mean */
};

/* Feature-major codebook block: out[(v-v0)*ld + (i-i0)] = W[v*M + i] for
 * v in [v0,v1), i in [i0,i1). The blurred kind needs M = E*E. */
int synth_codebook(uint64_t seed, int kind, int64_t V, int64_t M, int64_t v0, int64_t v1, int64_t i0,
                   int64_t i1, float *out, int64_t ld, int nthreads);

/* Row lengths 1 + Poisson(lam), capped at V, as a CSR row-pointer array of
 * N+1 entries starting at 0. Returns the total count, or <0 (-2: the total
 * exceeds int32). */
int64_t synth_csr_row_ptr(uint64_t seed, int64_t N, int64_t V, double lam, int32_t *row_ptr, int nthreads);

/* Fills each row with distinct feature ids drawn from Zipf(zipf_s) over ranks
 * 1..V (id = rank-1) without replacement, sorted ascending. row_ptr must come
 * from synth_csr_row_ptr with the same seed, N, V and lam. */
int synth_csr_col_idx(uint64_t seed, int64_t N, int64_t V, double lam, double zipf_s, const int32_t *row_ptr,
                      int32_t *col_idx, int nthreads);

/* Values of a sparse real-valued batch: out[q] for the ids at CSR positions
 * q = 0 .. n-1, each a pure function of (seed, q).
 *   SYNTH_VAL_UNIFORM    (h+1) * 2^-24 with 24 random bits h: in (0, 1]
 *   SYNTH_VAL_QUANTISED  (k+1) / 256 with k uniform on {0..255}: in [1/256, 1]
 * Returns 0, or -1 on bad arguments. */
enum { SYNTH_VAL_UNIFORM = 0, SYNTH_VAL_QUANTISED = 1 };
int synth_values(uint64_t seed, int kind, int64_t n, float *out, int nthreads);

/* Number of distinct feature ids in each group of TA consecutive rows
 * (the last group may be short): out has ceil(N/TA) entries. */
int synth_tile_distinct(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t TA, int32_t *out,
                        int nthreads);

#ifdef __cplusplus
}
#endif
#endif
