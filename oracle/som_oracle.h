/*
 * som_oracle.h -- CPU oracle for the sparse-binary BMU search.
 *
 * TEST INFRASTRUCTURE ONLY. The product library never includes, links or
 * calls this code; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do. It shares no code with the HIP path.
 *
 * It evaluates the definition of the best-matching unit (Method, problem
 * statement, Eq. (1)): for a sparse-binary input x over V features and a
 * codebook of prototypes w_i,
 *
 *     D_i = sum_{v=0}^{V-1} (x_v - w_{v,i})^2        (fp64, v ascending)
 *     bmu = lowest i with D_i = min_j D_j            (lowest-index tie-break,
 *                                                     problem statement)
 *
 * with x_v = 1 for the row's active feature ids and 0 elsewhere, over a
 * feature-major codebook (element (v, i) at W[v*ldw + (i - i0)], the layout
 * of the feature-major codebook section). One thread, no blocking.
 */
#ifndef SOM_ORACLE_H
#define SOM_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (0 = success). */
#define SOM_ORACLE_OK 0
#define SOM_ORACLE_BAD_ARG 1   /* null pointer, empty block, ldw too small, N<0, V<1 */
#define SOM_ORACLE_BAD_CSR 2   /* row_ptr negative or decreasing, or a feature id outside [0, V) */
#define SOM_ORACLE_NO_MEM 3

/*
 * Dense BMU over the neuron block [i0, i1) of a feature-major fp32 codebook.
 *   W        host, V rows of at least (i1-i0) floats, row stride ldw >= i1-i0;
 *            W[v*ldw + k] is the weight of feature v for neuron i0+k.
 *   row_ptr  host int32[N+1]; row s holds col_idx[row_ptr[s] .. row_ptr[s+1]).
 *            row_ptr[0] may be non-zero (col_idx is the base the offsets index).
 *   col_idx  host int32 feature ids in [0, V). A repeated id counts once (x is
 *            binary); order within a row does not matter.
 *   bmu      out int32[N]: global index (i0 + k) of the best unit.
 *   dist     out fp64[N]:  D_bmu, the full squared Euclidean distance.
 *   dist2    out fp64[N]:  min over i != bmu of D_i (+inf if the block holds
 *            one neuron). May be NULL.
 * Returns a SOM_ORACLE_* code; outputs are unspecified on error.
 */
int som_bmu_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                        const int32_t *col_idx, int64_t N, int32_t *bmu, double *dist, double *dist2);

/*
 * The two best units over the same block, in the order (D_i, i): smallest
 * distance first, the lower index first among equal distances (the tie-break
 * above applied to every rank). The paper's fused sweep returns the two best
 * units of each sample (Figure 2 caption); the second one defines the
 * topographic error (Background, quality measures).
 *   bmu, dist    rank 1, as som_bmu_oracle_host.
 *   bmu2, dist2  rank 2 (global index); -1 and +inf if the block holds one neuron.
 *   dist3        D of rank 3 (+inf if fewer than three neurons). May be NULL.
 */
int som_bmu2_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                         const int32_t *col_idx, int64_t N, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2,
                         double *dist3);

/*
 * Sparse real-valued inputs (Discussion: the gather-multiply variant, a values
 * array beside the feature ids): x_v = values[p] for the id col_idx[p] of the
 * row, 0 elsewhere, and D_i = sum_v (x_v - w_{v,i})^2 in fp64, v ascending.
 * Ranks and outputs as som_bmu2_oracle_host. values: host float[nnz], indexed
 * like col_idx.
 */
int som_bmu_sf_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, const int32_t *row_ptr,
                           const int32_t *col_idx, const float *values, int64_t N, int32_t *bmu, double *dist,
                           int32_t *bmu2, double *dist2, double *dist3);

/*
 * One batch-SOM update for binary rows (Algorithm 2, steps 8-9; the factorised
 * box-blur update section), on an E x E lattice, neuron i = row*E + col,
 * feature-major codebook W[v*M + i] with M = E*E.
 *   bmu     host int32[N], the best unit of every sample (from a search).
 *   radius  box half-width r >= 1 (the schedule's sigma rounded to whole cells,
 *           at least one).
 *   W_out   host float[V*M]: num/den clamped to [0, 1] where the unit has a
 *           sample within 3r cells along both axes and the blurred den > 0,
 *           else W_in.
 * num[v][i] = number of samples at unit i holding feature v, den[i] = number of
 * samples at unit i, both converted to fp32, then blurred: three box passes
 * along every lattice row, then three along every lattice column, each pass a
 * running window sum over the clamped window (first window summed in ascending
 * order, then add the element entering, subtract the one leaving), unnormalised,
 * in fp32; the quotient is an fp32 division. In exact arithmetic the blurred den
 * is zero exactly where no unit within 3r cells along both axes holds a sample
 * (three clamped windows of half-width r reach that far); fp32 running sums past
 * 2^24 can leave a residual there (or a wrong quotient near its edge), so units
 * outside that support -- counted exactly, in whole numbers -- keep W_in, and
 * quotients are clamped to [0, 1]. Plain loops, one thread.
 */
int som_update_oracle_host(const float *W_in, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx,
                           int64_t N, const int32_t *bmu, int64_t radius, float *W_out);

/*
 * Per-neuron squared norms n_i = sum_v w_{v,i}^2 in fp64, v ascending, for
 * i in [i0, i1): norms[i - i0]. Same W layout as above.
 */
int som_norms_oracle_host(const float *W, int64_t ldw, int64_t V, int64_t i0, int64_t i1, double *norms);

#ifdef __cplusplus
}
#endif
#endif
