/*
 * oracle.c -- plain CPU oracle for the sparse-binary BMU search.
 *
 * TEST INFRASTRUCTURE ONLY (see som_oracle.h): never linked into the product
 * library. Written from the paper's definition, not from any kernel:
 *
 *   - Eq. (1), problem statement: BMU(x) = argmin_i ||x - w_i||^2. The oracle
 *     evaluates the squared distance term by term over all V features, in
 *     fp64; it does not use the expanded form ||w||^2 - 2<x,w>.
 *   - Problem statement: ties go to the lowest neuron index; features are
 *     taken in ascending order (here: v = 0..V-1 for every neuron).
 *   - Feature-major codebook section: weight (v, i) sits at W[v*M + i].
 *
 *   - Figure 2 caption and the quality measures of the Background section:
 *     the two best units of every sample (the second feeds the topographic
 *     error). som_bmu2_oracle_host ranks units by (D_i, i) and returns the
 *     first two, plus the third distance for margin checks.
 *   - Discussion, sparse real-valued inputs: som_bmu_sf_oracle_host takes a
 *     value with every feature id (x_v real instead of 1) and ranks the same
 *     squared distance.
 *
 * The loops run feature-outer, neuron-inner. For each neuron the terms are
 * still added one at a time in ascending v, so every D_i is exactly the
 * value the neuron-outer loop would produce; the interchange only makes the
 * codebook stream in its storage order.
 */
#include "som_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static int check_args(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                      const int32_t *col_idx, int64_t N)
{
    if (N < 0 || V < 1 || i0 < 0 || i1 <= i0 || ldw < i1 - i0) return SOM_ORACLE_BAD_ARG;
    if (N == 0) return SOM_ORACLE_OK;
    if (!W || !row_ptr) return SOM_ORACLE_BAD_ARG;
    for (int64_t s = 0; s < N; ++s)
        if (row_ptr[s + 1] < row_ptr[s]) return SOM_ORACLE_BAD_CSR;
    if (row_ptr[N] > row_ptr[0] && !col_idx) return SOM_ORACLE_BAD_ARG;
    return SOM_ORACLE_OK;
}

/* x = the binary input vector of row s (x_v = 1 for its feature ids, 0 elsewhere). */
static int input_vector(const int32_t *row_ptr, const int32_t *col_idx, int64_t s, int64_t V, double *x)
{
    for (int64_t v = 0; v < V; ++v) x[v] = 0.0;
    for (int64_t p = row_ptr[s]; p < row_ptr[s + 1]; ++p) {
        const int32_t v = col_idx[p];
        if (v < 0 || v >= V) return SOM_ORACLE_BAD_CSR;
        x[v] = 1.0;
    }
    return SOM_ORACLE_OK;
}

/* x = the real-valued input vector of row s: x_v = the value given with id v, 0 elsewhere. */
static int input_values(const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t s, int64_t V,
                        double *x)
{
    for (int64_t v = 0; v < V; ++v) x[v] = 0.0;
    for (int64_t p = row_ptr[s]; p < row_ptr[s + 1]; ++p) {
        const int32_t v = col_idx[p];
        if (v < 0 || v >= V) return SOM_ORACLE_BAD_CSR;
        x[v] = (double)values[p];
    }
    return SOM_ORACLE_OK;
}

/* D_k = sum_v (x_v - w_{v,k})^2 for the block's neurons k = 0..B-1, v ascending. */
static void distances(const float *W, int64_t ldw, int64_t V, int64_t B, const double *x, double *D)
{
    for (int64_t k = 0; k < B; ++k) D[k] = 0.0;
    for (int64_t v = 0; v < V; ++v) {
        const float *wrow = W + v * ldw;
        for (int64_t k = 0; k < B; ++k) {
            const double diff = x[v] - (double)wrow[k];
            D[k] += diff * diff;
        }
    }
}

int som_bmu_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                        const int32_t *col_idx, int64_t N, int32_t *bmu, double *dist, double *dist2)
{
    int rc = check_args(W, ldw, V, i0, i1, row_ptr, col_idx, N);
    if (rc != SOM_ORACLE_OK || N == 0) return rc;
    if (!bmu || !dist) return SOM_ORACLE_BAD_ARG;

    const int64_t B = i1 - i0;
    double *D = (double *)malloc((size_t)B * sizeof(double));
    double *x = (double *)malloc((size_t)V * sizeof(double));
    if (!D || !x) {
        free(D);
        free(x);
        return SOM_ORACLE_NO_MEM;
    }

    for (int64_t s = 0; s < N; ++s) {
        if ((rc = input_vector(row_ptr, col_idx, s, V, x)) != SOM_ORACLE_OK) break;
        distances(W, ldw, V, B, x, D);

        /* argmin, lowest index among equal distances */
        int64_t best = 0;
        for (int64_t k = 1; k < B; ++k)
            if (D[k] < D[best]) best = k;
        /* second-best distance over the other neurons */
        double second = INFINITY;
        for (int64_t k = 0; k < B; ++k)
            if (k != best && D[k] < second) second = D[k];

        bmu[s] = (int32_t)(i0 + best);
        dist[s] = D[best];
        if (dist2) dist2[s] = second;
    }
    free(D);
    free(x);
    return rc;
}

int som_bmu2_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                         const int32_t *col_idx, int64_t N, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2,
                         double *dist3)
{
    int rc = check_args(W, ldw, V, i0, i1, row_ptr, col_idx, N);
    if (rc != SOM_ORACLE_OK || N == 0) return rc;
    if (!bmu || !dist || !bmu2 || !dist2) return SOM_ORACLE_BAD_ARG;

    const int64_t B = i1 - i0;
    double *D = (double *)malloc((size_t)B * sizeof(double));
    double *x = (double *)malloc((size_t)V * sizeof(double));
    if (!D || !x) {
        free(D);
        free(x);
        return SOM_ORACLE_NO_MEM;
    }

    for (int64_t s = 0; s < N; ++s) {
        if ((rc = input_vector(row_ptr, col_idx, s, V, x)) != SOM_ORACLE_OK) break;
        distances(W, ldw, V, B, x, D);

        /* The first three units in the order (D_k, k): scanning k upwards, a unit
         * moves ahead of a kept one only if its distance is strictly smaller. */
        int64_t r1 = -1, r2 = -1, r3 = -1;
        for (int64_t k = 0; k < B; ++k) {
            if (r1 < 0 || D[k] < D[r1]) {
                r3 = r2;
                r2 = r1;
                r1 = k;
            } else if (r2 < 0 || D[k] < D[r2]) {
                r3 = r2;
                r2 = k;
            } else if (r3 < 0 || D[k] < D[r3]) {
                r3 = k;
            }
        }
        bmu[s] = (int32_t)(i0 + r1);
        dist[s] = D[r1];
        bmu2[s] = r2 < 0 ? -1 : (int32_t)(i0 + r2);
        dist2[s] = r2 < 0 ? INFINITY : D[r2];
        if (dist3) dist3[s] = r3 < 0 ? INFINITY : D[r3];
    }
    free(D);
    free(x);
    return rc;
}

int som_bmu_sf_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                           const int32_t *col_idx, const float *values, int64_t N, int32_t *bmu, double *dist,
                           int32_t *bmu2, double *dist2, double *dist3)
{
    int rc = check_args(W, ldw, V, i0, i1, row_ptr, col_idx, N);
    if (rc != SOM_ORACLE_OK || N == 0) return rc;
    if (!bmu || !dist || !bmu2 || !dist2 || (row_ptr[N] > row_ptr[0] && !values)) return SOM_ORACLE_BAD_ARG;

    const int64_t B = i1 - i0;
    double *D = (double *)malloc((size_t)B * sizeof(double));
    double *x = (double *)malloc((size_t)V * sizeof(double));
    if (!D || !x) {
        free(D);
        free(x);
        return SOM_ORACLE_NO_MEM;
    }

    for (int64_t s = 0; s < N; ++s) {
        if ((rc = input_values(row_ptr, col_idx, values, s, V, x)) != SOM_ORACLE_OK) break;
        distances(W, ldw, V, B, x, D);

        /* the first three units in the order (D_k, k), as in som_bmu2_oracle_host */
        int64_t q1 = -1, q2 = -1, q3 = -1;
        for (int64_t k = 0; k < B; ++k) {
            if (q1 < 0 || D[k] < D[q1]) {
                q3 = q2;
                q2 = q1;
                q1 = k;
            } else if (q2 < 0 || D[k] < D[q2]) {
                q3 = q2;
                q2 = k;
            } else if (q3 < 0 || D[k] < D[q3]) {
                q3 = k;
            }
        }
        bmu[s] = (int32_t)(i0 + q1);
        dist[s] = D[q1];
        bmu2[s] = q2 < 0 ? -1 : (int32_t)(i0 + q2);
        dist2[s] = q2 < 0 ? INFINITY : D[q2];
        if (dist3) dist3[s] = q3 < 0 ? INFINITY : D[q3];
    }
    free(D);
    free(x);
    return rc;
}

int som_norms_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, double *norms)
{
    if (!W || !norms || V < 1 || i0 < 0 || i1 <= i0 || ldw < i1 - i0) return SOM_ORACLE_BAD_ARG;
    const int64_t B = i1 - i0;
    for (int64_t k = 0; k < B; ++k) norms[k] = 0.0;
    for (int64_t v = 0; v < V; ++v) {
        const float *wrow = W + v * ldw;
        for (int64_t k = 0; k < B; ++k) {
            const double w = (double)wrow[k];
            norms[k] += w * w;
        }
    }
    return SOM_ORACLE_OK;
}
