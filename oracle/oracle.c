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
 * The loops run feature-outer, neuron-inner. For each neuron the terms are
 * still added one at a time in ascending v, so every D_i is exactly the
 * value the neuron-outer loop would produce; the interchange only makes the
 * codebook stream in its storage order.
 */
#include "som_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

int som_bmu_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                        const int32_t *col_idx, int64_t N, int32_t *bmu, double *dist, double *dist2)
{
    if (N < 0 || V < 1 || i0 < 0 || i1 <= i0 || ldw < i1 - i0) return SOM_ORACLE_BAD_ARG;
    if (N == 0) return SOM_ORACLE_OK;
    if (!W || !row_ptr || !bmu || !dist) return SOM_ORACLE_BAD_ARG;
    for (int64_t s = 0; s < N; ++s)
        if (row_ptr[s + 1] < row_ptr[s]) return SOM_ORACLE_BAD_CSR;
    if (row_ptr[N] > row_ptr[0] && !col_idx) return SOM_ORACLE_BAD_ARG;

    const int64_t B = i1 - i0;
    double *D = (double *)malloc((size_t)B * sizeof(double));
    unsigned char *x = (unsigned char *)malloc((size_t)V);
    if (!D || !x) {
        free(D);
        free(x);
        return SOM_ORACLE_NO_MEM;
    }

    for (int64_t s = 0; s < N; ++s) {
        /* the binary input vector x of sample s */
        memset(x, 0, (size_t)V);
        for (int64_t p = row_ptr[s]; p < row_ptr[s + 1]; ++p) {
            const int32_t v = col_idx[p];
            if (v < 0 || v >= V) {
                free(D);
                free(x);
                return SOM_ORACLE_BAD_CSR;
            }
            x[v] = 1;
        }

        /* D_i = sum_v (x_v - w_{v,i})^2, v ascending */
        for (int64_t k = 0; k < B; ++k) D[k] = 0.0;
        for (int64_t v = 0; v < V; ++v) {
            const double xv = x[v] ? 1.0 : 0.0;
            const float *wrow = W + v * ldw;
            for (int64_t k = 0; k < B; ++k) {
                const double diff = xv - (double)wrow[k];
                D[k] += diff * diff;
            }
        }

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
    return SOM_ORACLE_OK;
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
