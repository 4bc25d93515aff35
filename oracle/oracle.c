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
 *   - Factorised box-blur section and Algorithm 2, steps 8-9: the batch update.
 *     som_update_oracle_host scatters the batch onto the lattice (per unit, the
 *     count of assigned samples and, per feature, of those holding it), blurs
 *     both fields with three running-sum box passes along the rows and three
 *     along the columns (clamped window, unnormalised, fp32 as the paper
 *     fixes), and divides, leaving units with no sample in their neighbourhood
 *     unchanged (a zero denominator, read on the exact support: see below) and
 *     keeping every quotient in [0, 1], the range of a mean of 0/1 inputs.
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
    if (row_ptr[0] < 0) return SOM_ORACLE_BAD_CSR; /* offsets index col_idx from its start */
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

/* ------------------------------------------------------------------ update */

/* One box pass over n values of a lattice line (stride apart), half-width r,
 * clamped: out[i] = sum of line[j] for |j - i| <= r, 0 <= j < n, kept as a
 * running window sum in fp32 -- the window's first sum in ascending j, then per
 * step the element entering is added and the one leaving subtracted. */
static void box_pass(float *line, int64_t n, int64_t stride, int64_t r, float *tmp)
{
    float s = 0.0f;
    for (int64_t j = 0; j <= r && j < n; ++j) s += line[j * stride];
    tmp[0] = s;
    for (int64_t i = 1; i < n; ++i) {
        if (i + r < n) s += line[(i + r) * stride];
        if (i - r - 1 >= 0) s -= line[(i - r - 1) * stride];
        tmp[i] = s;
    }
    for (int64_t i = 0; i < n; ++i) line[i * stride] = tmp[i];
}

/* Three passes along every lattice row, then three along every lattice column. */
/* sup[i] = occupied units (cnt > 0) within R cells of unit i along both lattice
 * axes (windows clamped to the lattice): window counts along every row, then
 * along every column, each from a prefix sum of whole numbers. */
static int occupied_support(const int64_t *cnt, int64_t E, int64_t R, int64_t *sup)
{
    int64_t *pre = (int64_t *)malloc((size_t)(E + 1) * sizeof(int64_t));
    if (!pre) return SOM_ORACLE_NO_MEM;
    for (int64_t row = 0; row < E; ++row) {
        pre[0] = 0;
        for (int64_t c = 0; c < E; ++c) pre[c + 1] = pre[c] + (cnt[row * E + c] > 0 ? 1 : 0);
        for (int64_t c = 0; c < E; ++c) {
            const int64_t lo = c - R < 0 ? 0 : c - R, hi = c + R + 1 > E ? E : c + R + 1;
            sup[row * E + c] = pre[hi] - pre[lo];
        }
    }
    for (int64_t c = 0; c < E; ++c) {
        pre[0] = 0;
        for (int64_t row = 0; row < E; ++row) pre[row + 1] = pre[row] + sup[row * E + c];
        for (int64_t row = 0; row < E; ++row) {
            const int64_t lo = row - R < 0 ? 0 : row - R, hi = row + R + 1 > E ? E : row + R + 1;
            sup[row * E + c] = pre[hi] - pre[lo];
        }
    }
    free(pre);
    return SOM_ORACLE_OK;
}

static void blur_field(float *f, int64_t E, int64_t r, float *tmp)
{
    for (int64_t row = 0; row < E; ++row)
        for (int pass = 0; pass < 3; ++pass) box_pass(f + row * E, E, 1, r, tmp);
    for (int64_t col = 0; col < E; ++col)
        for (int pass = 0; pass < 3; ++pass) box_pass(f + col, E, E, r, tmp);
}

int som_update_oracle_host(const float *W_in, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx,
                           int64_t N, const int32_t *bmu, int64_t radius, float *W_out)
{
    if (!W_in || !W_out || V < 1 || E < 1 || N < 0 || radius < 1 || (N > 0 && (!row_ptr || !bmu)))
        return SOM_ORACLE_BAD_ARG;
    const int64_t M = E * E;
    if (N > 0 && row_ptr[0] < 0) return SOM_ORACLE_BAD_CSR;
    for (int64_t s = 0; s < N; ++s) {
        if (row_ptr[s + 1] < row_ptr[s]) return SOM_ORACLE_BAD_CSR;
        if (bmu[s] < 0 || bmu[s] >= M) return SOM_ORACLE_BAD_ARG;
    }
    if (N > 0 && row_ptr[N] > row_ptr[0] && !col_idx) return SOM_ORACLE_BAD_ARG;

    int64_t *cnt = (int64_t *)calloc((size_t)M, sizeof(int64_t));
    int64_t *sup = (int64_t *)calloc((size_t)M, sizeof(int64_t));
    float *den = (float *)malloc((size_t)M * sizeof(float));
    float *num = (float *)malloc((size_t)M * sizeof(float));
    float *tmp = (float *)malloc((size_t)E * sizeof(float));
    int rc = SOM_ORACLE_OK;
    if (!cnt || !sup || !den || !num || !tmp) {
        rc = SOM_ORACLE_NO_MEM;
        goto done;
    }

    /* den: samples per unit (Algorithm 2, step 8), blurred */
    for (int64_t s = 0; s < N; ++s) cnt[bmu[s]] += 1;
    for (int64_t i = 0; i < M; ++i) den[i] = (float)cnt[i];
    blur_field(den, E, radius, tmp);
    /* Where the blurred denominator is zero in exact arithmetic: no occupied unit
     * within 3*radius cells along both axes (three windows of half-width radius,
     * clamped to the lattice, reach exactly that far). fp32 running sums that pass
     * 2^24 can leave a residual there, so the keep-the-prototype rule is taken on
     * this support, counted in whole numbers. */
    if ((rc = occupied_support(cnt, E, 3 * radius, sup)) != SOM_ORACLE_OK) goto done;

    /* num, one feature at a time: samples per unit holding feature v (x binary) */
    for (int64_t v = 0; v < V; ++v) {
        for (int64_t i = 0; i < M; ++i) cnt[i] = 0;
        for (int64_t s = 0; s < N; ++s)
            for (int64_t p = row_ptr[s]; p < row_ptr[s + 1]; ++p) {
                if (col_idx[p] < 0 || col_idx[p] >= V) {
                    rc = SOM_ORACLE_BAD_CSR;
                    goto done;
                }
                if (col_idx[p] == v) cnt[bmu[s]] += 1;
            }
        for (int64_t i = 0; i < M; ++i) num[i] = (float)cnt[i];
        blur_field(num, E, radius, tmp);
        /* the prototype becomes the neighbourhood mean, a mean of 0/1 inputs and so in
         * [0, 1] (the quotient of rounded sums is clamped there); a unit with no sample
         * in its neighbourhood, or whose rounded denominator is not positive, keeps its
         * prototype */
        for (int64_t i = 0; i < M; ++i) {
            if (sup[i] > 0 && den[i] > 0.0f) {
                const float q = num[i] / den[i];
                W_out[v * M + i] = fminf(fmaxf(q, 0.0f), 1.0f);
            } else {
                W_out[v * M + i] = W_in[v * M + i];
            }
        }
    }
done:
    free(sup);
    free(cnt);
    free(den);
    free(num);
    free(tmp);
    return rc;
}
