/*
 * som.h -- C ABI of libsom.so, the MI355X (gfx950) best-matching-unit search
 * for sparse-binary self-organising maps.
 *
 * What it computes (Method, problem statement, Eq. (1)): for every
 * sparse-binary input x -- the sorted set of its active feature ids -- and a
 * codebook of M prototypes w_i over V features stored feature-major
 * (W[v*M + i], Method, feature-major codebook),
 *
 *     BMU(x) = argmin_i ||x - w_i||^2 = argmin_i ( ||w_i||^2 - 2 <x, w_i> ),
 *     <x, w_i> = sum over the active features v of W[v*M + i]   (a gather-sum),
 *
 * ties going to the lowest neuron index (problem statement). The search is
 * the tiled sweep of the SpMM-tile kernel section (Algorithm 2, steps 4-7):
 * samples are grouped into tiles, each codebook row a tile touches is read
 * once and added into every sample of the tile that holds that feature, and
 * the argmin is taken inside the sweep, so no N x M score block is ever
 * written.
 *
 * Numerics. Norms ||w_i||^2 are fp64 sums in ascending feature order. Each
 * sample's dot product is an fp32 sum of its weights in ascending feature
 * order, whatever the tile size. The ranked value is the fp64
 * d_i = ||w_i||^2 - 2*dot_i (one rounding). The argmin compares 64-bit keys:
 * the top 44 bits of an order-preserving image of d_i's fp64 pattern, then
 * the 20-bit neuron index (so M <= 2^20); two values within about 2^-32 of
 * each other (relative) compare by index. The returned distance is the full
 * squared Euclidean distance ||x - w_bmu||^2 = d_bmu + nnz(x), in fp64.
 *
 * Conventions for every entry point:
 *   - Pointers documented "device" are HIP device memory of the current
 *     device (torch tensors' data_ptr() on ROCm); "host" pointers are
 *     ordinary host memory.
 *   - `stream` is a hipStream_t (NULL = the default stream). Device work is
 *     enqueued on it and the call returns without waiting; inputs must stay
 *     alive and outputs must not be read until the stream has synchronised.
 *   - The caller owns every buffer. No entry point allocates device memory:
 *     scratch space comes from the caller's workspace.
 *   - Calls on different workspaces and streams may run concurrently.
 *   - Cheap argument checks run on the host before anything is enqueued; on
 *     failure nothing is enqueued and a status other than SOM_OK is returned,
 *     with a description available from som_last_error() on the same thread.
 *   - No C++ exception crosses the ABI. N == 0 is a valid no-op.
 *
 * CSR input. row_ptr has N+1 int32 entries; row s holds the feature ids
 * col_idx[row_ptr[s] .. row_ptr[s+1]). row_ptr[0] need not be 0 (a slice of
 * a larger batch) but must not be negative: col_idx is always the base
 * pointer the offsets index, and nnz = row_ptr[N] - row_ptr[0] (the device
 * reads a batch whose row_ptr[0] is negative as empty and flags it). Each
 * row's ids must be strictly ascending
 * and in [0, V) (sorted, distinct: the paper's sparse-binary CSR, corpus
 * section). That is a precondition of the device path, checked on the host
 * by som_validate_csr_host. The device kernels never access memory outside
 * the buffers they are given, whatever the CSR holds; a violation they see
 * is recorded in the workspace and reported by som_bmu_input_flags, and the
 * results of the affected samples are then unspecified.
 */
#ifndef SOM_H
#define SOM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SOM_OK = 0,
    SOM_ERR_INVALID_ARG = 1, /* null pointer, negative or oversized dimension, bad config */
    SOM_ERR_BAD_CSR = 2,     /* (som_validate_csr_host) the CSR breaks the input rules above */
    SOM_ERR_WORKSPACE = 3,   /* workspace too small or misaligned */
    SOM_ERR_HIP = 4          /* a HIP runtime call or launch failed */
} som_status;

/* Largest map the 20-bit index field of the argmin key can address. */
#define SOM_MAX_NEURONS (1 << 20)

/* Bits reported by som_bmu_input_flags. A flagged batch breaks the CSR
 * preconditions; its results are defined only as far as stated here: an id
 * outside [0, V) is left out of the row's dot products (the binary row's
 * ||x||^2, its length, still counts it), and rows with valid ids get the
 * results they get in a valid batch. Rows with unsorted or repeated ids get
 * in-range but unspecified results. Row pointers are checked before any row
 * is read: a batch whose row_ptr decreases or leaves [row_ptr[0],
 * row_ptr[0] + nnz] is searched as if every row were empty (each sample gets
 * the unit of smallest norm, lowest index first; its distance is unspecified
 * when the batch is not regrouped), so overlapping rows cannot multiply the
 * work. No input drives an access out of bounds. */
#define SOM_FLAG_ID_RANGE 0x1u   /* a feature id outside [0, V) was skipped      */
#define SOM_FLAG_UNSORTED 0x2u   /* a row's ids were not strictly ascending       */
#define SOM_FLAG_ROW_PTR 0x4u    /* row_ptr decreased or left [row_ptr[0], +nnz]  */

/*
 * Optional tuning of the search. Pass NULL for the defaults. Neither field
 * changes any result: a sample's sum order is fixed by its own features, so
 * its BMU and distance do not depend on the tile it lands in.
 *   tile_samples  samples per tile, TA (SpMM-tile kernel section): 8, 16 or
 *                 32; 0 selects SOM_DEFAULT_TILE_SAMPLES.
 *   keep_order    0 (default): the plan first regroups the batch by each
 *                 sample's least frequent feature (the post-submission
 *                 section's lever of clustering samples so tiles share
 *                 features), which shrinks tile unions and keeps rare
 *                 codebook rows in cache; results still come out in input
 *                 order. 1: tile the samples in the order given.
 * The same config must be given to the workspace query and to every phase
 * of one search.
 */
#define SOM_DEFAULT_TILE_SAMPLES 8

typedef struct {
    int32_t tile_samples;
    int32_t keep_order;
    int32_t reserved[6]; /* must be zero */
} som_bmu_config;

/*
 * Workspace bytes a search over N samples with nnz ids in total, on a map of
 * M neurons and V features, needs under `config` (NULL = defaults). Pure
 * host function; returns 0 if a size is out of range (see som_bmu_search)
 * or the config is invalid. The workspace must be 256-byte aligned device
 * memory. It holds the tile plan (8 bytes per id), one 8-byte partial key
 * and one 4-byte dot product per sample and strip of 512 neurons (256 when
 * tile_samples > 8) and, unless keep_order is set, the regrouped batch and
 * its staged results (4 bytes per id, 28 per sample, 12 per feature).
 */
size_t som_bmu_workspace_bytes(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config);

/*
 * Per-neuron squared norms (Algorithm 2, step 6; the separate norm pass of
 * the profiling section): norms[i] = sum_{v=0}^{V-1} W[v*M+i]^2, each square
 * formed exactly in fp64 and added in ascending v.
 *   W      device fp32, V*M elements, feature-major, 4-byte aligned.
 *   norms  device fp64 [M], written.
 * Run once per codebook; the result serves every later search on it.
 */
som_status som_codebook_norms(const float *W, int64_t V, int64_t M, double *norms, void *stream);

/*
 * BMU search over a CSR batch (Eq. (1); Algorithm 2, steps 4-7).
 *   W          device fp32 [V*M] feature-major codebook.
 *   norms      device fp64 [M] from som_codebook_norms on the same W.
 *   row_ptr    device int32 [N+1]; col_idx device int32 (see CSR input).
 *   nnz        row_ptr[N] - row_ptr[0], as the caller knows it (sizes the
 *              plan inside the workspace; the kernels never read past it).
 *   bmu        device int32 [N], written: index of the best unit.
 *   dist       device fp64 [N], written: ||x_s - w_bmu||^2.
 *   workspace  device, >= som_bmu_workspace_bytes(N, M, V, nnz, config)
 *              bytes, 256-byte aligned; its contents are scratch.
 *   config     NULL or a som_bmu_config (host memory, read during the call).
 * Equivalent to som_bmu_plan, som_bmu_sweep, som_bmu_finalize in order.
 */
som_status som_bmu_search(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                          const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                          void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream);

/*
 * som_bmu_search without a workspace argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation). Arguments, results and errors are those
 * of som_bmu_search; the scratch space is a device array inside the library,
 * SOM_NOALLOC_SCRATCH_BYTES on every GPU the library runs on, held until the
 * process ends. The call allocates nothing. A search whose
 * som_bmu_workspace_bytes(N, M, V, nnz, config) exceeds that size returns
 * SOM_ERR_WORKSPACE (checked on the host, nothing enqueued): at 12 ids per
 * row and V = 30,000 that is about 248,000 rows on a 64x64 map, 39,000 on a
 * 256x256 map and 2,700 on a 1024x1024 map.
 * The stream must belong to the calling thread's current device.
 * All calls on one GPU share its array: calls that overlap in time on one
 * GPU (other streams, other threads) race and give undefined results.
 */
#define SOM_NOALLOC_SCRATCH_BYTES (64u << 20)

som_status som_bmu_search_noalloc(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                                  const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                                  const som_bmu_config *config, void *stream);

/*
 * The three phases of som_bmu_search, for callers that time or overlap them.
 * Arguments mean the same as above; each phase reads what the previous one
 * left in the same workspace, so they must run in this order on one stream.
 *
 * som_bmu_plan -- tile plan (Algorithm 2, step 5; SpMM-tile kernel section):
 *   unless keep_order is set, the batch is first regrouped by each sample's
 *   least frequent feature (a permutation and its row offsets in the workspace;
 *   the rows are read from row_ptr / col_idx through it); then, for each
 *   tile of tile_samples consecutive rows, the ascending list of the distinct
 *   feature ids its rows hold, each with a bit mask of the rows holding it.
 *   Also clears and sets the input flags.
 */
som_status som_bmu_plan(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz, int64_t V,
                        int64_t M, void *workspace, size_t workspace_bytes, const som_bmu_config *config,
                        void *stream);

/*
 * som_bmu_sweep -- the fused sweep (Algorithm 2, steps 4, 6, 7): streams each
 *   planned codebook row once per tile and neuron strip, accumulates every
 *   sample's dot product in registers, ranks d_i = ||w_i||^2 - 2*dot_i and
 *   keeps, per sample and group of neurons, the smallest 64-bit key and the
 *   fp32 dot product of the neuron it names.
 */
som_status som_bmu_sweep(const float *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                         void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream);

/*
 * som_bmu_finalize -- reduces the per-strip keys of each sample to its BMU
 *   and forms the winner's full squared distance from the dot product the
 *   sweep kept with the winning key: dist = (||w_bmu||^2 - 2*dot) + nnz(x).
 *   Reads only the workspace, norms and row_ptr (for nnz(x)); writes bmu and
 *   dist.
 */
som_status som_bmu_finalize(const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N, int64_t nnz,
                            int32_t *bmu, double *dist, void *workspace, size_t workspace_bytes,
                            const som_bmu_config *config, void *stream);

/*
 * The two best units per sample in the same fused sweep (SpMM-tile kernel
 * section, Figure 2 caption; the pair defines the topographic error of the
 * quality measures). Units are ranked by their distance, then by index:
 *   bmu, dist    as som_bmu_search.
 *   bmu2, dist2  device int32 [N] / fp64 [N], written: the next unit in that
 *                order and its full squared distance; -1 and +inf if M == 1.
 * The workspace must hold som_bmu2_workspace_bytes(N, M, V, nnz, config)
 * bytes: the single-best workspace plus a second key and dot product per
 * sample and strip (and, unless keep_order is set, 16 bytes per sample for
 * the staged second results). A two-best workspace also serves every single-best call
 * and som_bmu_input_flags with the same config.
 */
size_t som_bmu2_workspace_bytes(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config);

som_status som_bmu2_search(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                           const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2,
                           double *dist2, void *workspace, size_t workspace_bytes, const som_bmu_config *config,
                           void *stream);

/*
 * Its phases: som_bmu_plan (shared with the single-best search), then
 *   som_bmu2_sweep -- the fused sweep keeping, per sample and strip, the two
 *     smallest keys and their neurons' dot products;
 *   som_bmu2_finalize -- the two smallest keys over the strips, with their
 *     full squared distances.
 * Same arguments and ordering rules as the single-best phases, on a two-best
 * workspace.
 */
som_status som_bmu2_sweep(const float *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                          void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream);

som_status som_bmu2_finalize(const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N,
                             int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2, void *workspace,
                             size_t workspace_bytes, const som_bmu_config *config, void *stream);

/*
 * FP16 codebook storage (feature-major codebook section: the codebook is held
 * in IEEE half precision and widened to fp32 only for the accumulation, which
 * halves the bytes each codebook row costs). W holds
 * V*M IEEE binary16 bit patterns, feature-major as above, 2-byte aligned
 * (16-byte alignment and M a multiple of 8 select the vector loads). Every
 * other argument, the workspace and the results are those of the fp32 entry
 * point of the same name: the search on an fp16 codebook returns exactly what
 * the fp32 search returns on the same values widened to fp32 (the widening
 * and the squares are exact), so the oracle and the bars are unchanged.
 */
som_status som_codebook_norms_f16(const uint16_t *W, int64_t V, int64_t M, double *norms, void *stream);

som_status som_bmu_search_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                              const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                              void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream);

som_status som_bmu_sweep_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                             void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream);

som_status som_bmu2_search_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                               const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                               int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                               const som_bmu_config *config, void *stream);

som_status som_bmu2_sweep_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                              void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream);

/*
 * Sparse real-valued rows (the Discussion's gather-multiply variant: a values
 * array beside the feature ids, and ||x||^2). values: device float [nnz],
 * indexed like col_idx (values[p] belongs to feature col_idx[p]), finite.
 * The BMU of x is argmin_i ||x - w_i||^2 with x_v the given values; the sweep
 * accumulates x_v * W[v*M+i] with one fp32 fused multiply-add per term in
 * ascending feature order, and dist = (||w||^2 - 2*dot) + ||x||^2 with
 * ||x||^2 the fp64 sum of the squared values in row order.
 *   bmu2, dist2  both NULL: the best unit only; both non-NULL: the two best,
 *                as som_bmu2_search.
 * Tiles of 8 samples only (tile_samples 0 or 8; other values are rejected).
 * The workspace (som_bmu_sf_workspace_bytes) adds 32 bytes per id for the
 * plan's per-entry values and 8 per sample for ||x||^2 to the two-best one.
 * With all values 1 the results equal the binary search's bit for bit.
 */
size_t som_bmu_sf_workspace_bytes(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config);

som_status som_bmu_sf_search(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                             const int32_t *col_idx, const float *values, int64_t N, int64_t nnz, int32_t *bmu,
                             double *dist, int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                             const som_bmu_config *config, void *stream);

som_status som_bmu_sf_search_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                                 const int32_t *col_idx, const float *values, int64_t N, int64_t nnz, int32_t *bmu,
                                 double *dist, int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                                 const som_bmu_config *config, void *stream);

/*
 * Phases of som_bmu_sf_search, in this order on one stream and workspace:
 *   som_bmu_sf_plan -- the plan with each entry's sample values and ||x||^2;
 *   som_bmu_sf_sweep(_f16) -- the sweep; two_best != 0 keeps the two best;
 *   som_bmu_sf_finalize -- as above (bmu2/dist2 non-NULL after a two-best sweep).
 */
som_status som_bmu_sf_plan(const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N,
                           int64_t nnz, int64_t V, int64_t M, void *workspace, size_t workspace_bytes,
                           const som_bmu_config *config, void *stream);

som_status som_bmu_sf_sweep(const float *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                            int32_t two_best, void *workspace, size_t workspace_bytes, const som_bmu_config *config,
                            void *stream);

som_status som_bmu_sf_sweep_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                                int32_t two_best, void *workspace, size_t workspace_bytes,
                                const som_bmu_config *config, void *stream);

som_status som_bmu_sf_finalize(const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N,
                               int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2, void *workspace,
                               size_t workspace_bytes, const som_bmu_config *config, void *stream);

/*
 * The batch-SOM update for binary rows (Algorithm 2, steps 8-9; the factorised
 * box-blur update section), in place on the codebook W (fp32, or binary16 for
 * som_update_f16), lattice E x E with neuron i = row*E + col (M = E*E).
 *   bmu             device int32 [N]: each sample's best unit (from a search on
 *                   the same batch; values outside [0, M) are skipped).
 *   radius          box half-width r >= 1: som_radius(som_sigma(epoch, ...)).
 *   chunk_features  features blurred per pass (0 = all V); the workspace holds
 *                   three chunk x M fields, so smaller chunks need less memory.
 * som_update_workspace_bytes(V, E, N, chunk_features) sizes the workspace for a
 * batch of N samples (three chunk x M fields, ten M-sized buffers and N int32
 * positions for sorting the samples of crowded units); 0 for invalid sizes.
 * Per unit, den = samples assigned to it and num[v] = those holding feature v
 * (exact integer counts), both converted to fp32 and blurred by three
 * running-sum box passes along every lattice row and then three along every
 * column, each over the clamped window [k-r, k+r] and unnormalised (the paper's
 * four rules: unnormalised sums, clamped boundary, a unit whose blurred den is
 * zero keeps its prototype, fp32 accumulation with the binary16 conversion only
 * at the final write). W = num / den, clamped to [0, 1] (the range of a mean of
 * 0/1 inputs). The blurred den is zero, in exact arithmetic, exactly where no
 * unit within 3r cells along both axes holds a sample; fp32 sums past 2^24 can
 * leave a residual there, so the keep-the-prototype rule is applied on that
 * support, counted exactly (and wherever the fp32 den is not positive). The
 * passes run in a fixed order, so the result is the same bits on every run.
 * Norms must be recomputed afterwards. N == 0 is a no-op. The row pointers
 * are checked on the device before any row is read: if row_ptr[0] is
 * negative, or row_ptr decreases or leaves [row_ptr[0], row_ptr[0] + nnz],
 * the codebook is left unchanged (som_validate_csr_host checks the rest of
 * the CSR rules; ids outside [0, V) are skipped).
 */
size_t som_update_workspace_bytes(int64_t V, int64_t E, int64_t N, int64_t chunk_features);

som_status som_update(float *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx, int64_t N,
                      int64_t nnz, const int32_t *bmu, int32_t radius, int64_t chunk_features, void *workspace,
                      size_t workspace_bytes, void *stream);

som_status som_update_f16(uint16_t *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx, int64_t N,
                          int64_t nnz, const int32_t *bmu, int32_t radius, int64_t chunk_features, void *workspace,
                          size_t workspace_bytes, void *stream);

/*
 * The neighbourhood schedule (factorised box-blur section: an exponential
 * endpoint schedule from sigma0 = 0.5*E towards sigma_min, rate 0.3), read as
 * sigma(e) = sigma_min + (sigma0 - sigma_min) * exp(-rate * (e - 1)) for epochs
 * e = 1, 2, ... (e < 1 is taken as 1), and the box half-width it gives: sigma
 * rounded to the nearest whole cell (halves up), never below 1. Host functions.
 */
double som_sigma(int32_t epoch, double sigma0, double sigma_min, double rate);
int32_t som_radius(double sigma);

/*
 * Input flags (SOM_FLAG_*) the last plan on this workspace recorded. Waits
 * for `stream`, then copies one word to *flags (host). 0 means the device
 * saw a valid CSR.
 */
som_status som_bmu_input_flags(const void *workspace, size_t workspace_bytes, int64_t N, int64_t M, int64_t V,
                               int64_t nnz, const som_bmu_config *config, uint32_t *flags, void *stream);

/*
 * Host check of the CSR input rules (corpus section: sorted descriptor ids
 * per row; binary values implicit): row_ptr[0] >= 0, row_ptr non-decreasing,
 * every id in [0, V), ids strictly ascending within each row. Host pointers; col_idx
 * may be NULL when row_ptr[N] == row_ptr[0]. Returns SOM_OK, SOM_ERR_BAD_CSR
 * (with the first offending row in som_last_error) or SOM_ERR_INVALID_ARG.
 */
som_status som_validate_csr_host(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t V);

/* Text describing the last failure on the calling thread ("" if none). */
const char *som_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
