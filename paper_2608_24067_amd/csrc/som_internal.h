// som_internal.h -- shared between the C-ABI layer and the kernels of libsom.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "som.h"

namespace som {

// Tile sizes (samples per tile) the library is built for, and the default.
constexpr int kDefaultTileSamples = SOM_DEFAULT_TILE_SAMPLES;
inline bool valid_tile(int ta) { return ta == 8 || ta == 16 || ta == 32; }

// Neurons per lane of the sweep: 8 (two 16-byte loads per codebook row) for tiles of 8
// samples, 4 for larger tiles, so that the TA x NPL register accumulators stay at
// 64 or 128 VGPRs. One wave covers a strip of 64 * NPL neurons.
inline int neurons_per_lane(int ta) { return ta <= 8 ? 8 : 4; }
inline int64_t strip_neurons(int ta) { return 64 * neurons_per_lane(ta); }
inline int64_t n_strips(int64_t M, int ta) { return (M + strip_neurons(ta) - 1) / strip_neurons(ta); }
inline int64_t n_tiles(int64_t N, int ta) { return (N + ta - 1) / ta; }

// One position's result of a regrouped batch, staged in the workspace: a whole 16-byte
// record, so the finalize writes full lines and the move back to input order reads one
// record per sample.
struct alignas(16) Staged {
    double d;
    int32_t b;
    int32_t pad;
};

// Workspace carve-up (offsets in bytes from the workspace base; every section 256-byte aligned).
// The order sections are empty when the caller keeps the given sample order.
struct Layout {
    size_t flags;   // uint32 [64]: input flags
    size_t plan;    // uint2 [nnz]: (feature id, sample mask) of every tile's union, tile t at its CSR offset
    size_t tiles;   // int2 [n_tiles]: (plan offset, union size) per tile
    size_t keys;    // uint64 [n_strips * N]: per-strip partial argmin keys, strip-major, by batch position
    size_t dots;    // float [n_strips * N]: fp32 dot product of the neuron each key names
    size_t freq;    // uint32 [V+1]: feature counts of the batch
    size_t bucket;  // uint64 [V+1]: per-bucket (samples << 32 | ids) counts, then offsets
    size_t skey;    // int32 [N]: each sample's bucket
    size_t rank;    // uint64 [N]: each sample's rank in its bucket (samples << 32 | ids before it)
    size_t inv;     // int32 [N]: each sample's position in the ordered batch (-1: never placed)
    size_t pos;     // int32 [2N+2]: per position p of the ordered batch, pos[2p] = its row offset and
                    // pos[2p+1] = where its ids start in the caller's col_idx; pos[2N] = all ids
    size_t res;     // Staged [N]: best unit and distance by position, before they go back to input order
    size_t keys2;   // uint64 [n_strips * N]: per-strip second-smallest keys (two-best search only)
    size_t dots2;   // float [n_strips * N]: their dot products (two-best search only)
    size_t res2;    // Staged [N]: second unit and distance by position (two-best search, ordered batch only)
    size_t vals;    // float [nnz * TA]: sample values of every plan entry (real-valued rows only)
    size_t xsq;     // double [N]: ||x||^2 by batch position (real-valued rows only)
    size_t total;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The two-best sections follow the single-best ones and the real-valued sections
// follow those, so each smaller layout is a prefix of the larger ones.
inline Layout layout_for(int64_t N, int64_t M, int64_t V, int64_t nnz, int ta, bool order, bool top2 = false,
                         bool real = false)
{
    Layout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align256(bytes);
        return at;
    };
    L.flags = take(256);  // first, so that its place does not depend on the sizes or the config
    L.plan = take((size_t)nnz * 8);
    L.tiles = take((size_t)n_tiles(N, ta) * 8);
    L.keys = take((size_t)n_strips(M, ta) * (size_t)N * 8);
    L.dots = take((size_t)n_strips(M, ta) * (size_t)N * 4);
    const size_t o = order ? 1 : 0;
    L.freq = take(o * (size_t)(V + 1) * 4);
    L.bucket = take(o * (size_t)(V + 1) * 8);
    L.skey = take(o * (size_t)N * 4);
    L.rank = take(o * (size_t)N * 8);
    L.inv = take(o * (size_t)N * 4);
    L.pos = take(o * (size_t)(N + 1) * 8);
    L.res = take(o * (size_t)N * sizeof(Staged));
    const size_t t2 = top2 ? 1 : 0;
    L.keys2 = take(t2 * (size_t)n_strips(M, ta) * (size_t)N * 8);
    L.dots2 = take(t2 * (size_t)n_strips(M, ta) * (size_t)N * 4);
    L.res2 = take(t2 * o * (size_t)N * sizeof(Staged));
    const size_t r = real ? 1 : 0;
    L.vals = take(r * (size_t)nnz * (size_t)ta * 4);
    L.xsq = take(r * (size_t)N * 8);
    L.total = off;
    return L;
}

struct OrderBuffers {
    uint32_t *freq;
    unsigned long long *bucket, *rank;
    int32_t *skey, *inv, *pos;
    Staged *res, *res2;  // results by position (res2: two-best only)
};

// Where the sweep leaves its per-(sample, strip) results.
struct SweepOut {
    unsigned long long *keys;
    float *dots;
    unsigned long long *keys2;  // two-best only, else null
    float *dots2;
};

// Records the calling thread's error text (som_last_error) and returns st.
som_status set_error(som_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

// Kernel launchers (som_kernels.hip). Each returns the launch's hipError_t.
hipError_t launch_norms(const float *W, int64_t V, int64_t M, double *norms, hipStream_t st);
// fp16 codebooks: W holds IEEE binary16 bit patterns.
hipError_t launch_norms_f16(const uint16_t *W, int64_t V, int64_t M, double *norms, hipStream_t st);
hipError_t launch_clear_flags(uint32_t *flags, hipStream_t st);
// Flags SOM_FLAG_ROW_PTR when row_ptr decreases or leaves [row_ptr[0], row_ptr[0] + nnz];
// the plan then reads the batch as empty.
hipError_t launch_check_rows(const int32_t *row_ptr, int64_t N, int64_t nnz, uint32_t *flags, hipStream_t st);
// values, vals, xsq: real-valued rows only (else null). row_ptr, col_idx, values: the caller's batch.
// ob non-null: the batch was regrouped: position p's row has plan offsets ob->pos[2p] ... and its
// ids start at ob->pos[2p + 1] in the caller's col_idx.
hipError_t launch_plan(int ta, const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N,
                       int64_t nnz, int64_t V, const OrderBuffers *ob, uint2 *plan, int2 *tiles, float *vals,
                       double *xsq, uint32_t *flags, hipStream_t st);
// f16: W holds binary16 values; top2: fill keys2/dots2 too; vals: real-valued rows (tile 8 only).
hipError_t launch_sweep(int ta, bool f16, bool top2, const void *W, const double *norms, int64_t M, int64_t N,
                        int64_t V, int64_t nnz, const uint2 *plan, const int2 *tiles, const float *vals,
                        const SweepOut &o, hipStream_t st);
// bmu2/dist2 non-null: the two best units. xsq: real-valued rows (else ||x||^2 = nnz of the row).
// ob non-null: the batch was regrouped (the row lengths come from ob->pos, not row_ptr); results
// are staged by position and then moved to their samples.
hipError_t launch_finalize(int ta, const double *norms, int64_t M, const int32_t *row_ptr, int64_t N, int64_t nnz,
                           const OrderBuffers *ob, const double *xsq, const SweepOut &o, int32_t *bmu, double *dist,
                           int32_t *bmu2, double *dist2, hipStream_t st);
hipError_t launch_order(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz, int64_t V,
                        const OrderBuffers &ob, uint32_t *flags, hipStream_t st);

// ----------------------------------------------------------------- update

// Workspace of the batch update (som_update.hip): the den field (counts and two
// float buffers, M each), the sort of heavy units' samples (start[M + 2],
// cursor[M], slot[M], hunit[M], order[N]) and, for one chunk of features, counts
// and two float buffers of chunk * M.
struct UpdateBuffers {
    uint32_t *flags;  // SOM_FLAG_ROW_PTR: the batch's row pointers are invalid, nothing is updated
    int32_t *den_cnt;
    int32_t *sup_row, *sup;  // the exact support of the blurred den (row windows, then both axes)
    float *den_a, *den_b;  // scratch of the den blur
    float *den_blur;       // the blurred den
    int32_t *start, *cursor, *slot, *hunit, *order;
    int32_t *cnt;
    float *a, *b;
};

struct UpdateLayout {
    size_t flags, den_cnt, sup_row, sup, den_a, den_b, den_blur, start, cursor, slot, hunit, order, cnt, a, b, total;
};

inline UpdateLayout update_layout(int64_t M, int64_t N, int64_t chunk)
{
    UpdateLayout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align256(bytes);
        return at;
    };
    L.flags = take(256);
    L.den_cnt = take((size_t)M * 4);
    L.sup_row = take((size_t)M * 4);
    L.sup = take((size_t)M * 4);
    L.den_a = take((size_t)M * 4);
    L.den_b = take((size_t)M * 4);
    L.den_blur = take((size_t)M * 4);
    L.start = take((size_t)(M + 2) * 4);
    L.cursor = take((size_t)M * 4);
    L.slot = take((size_t)M * 4);
    L.hunit = take((size_t)M * 4);
    L.order = take((size_t)N * 4);
    L.cnt = take((size_t)chunk * (size_t)M * 4);
    L.a = take((size_t)chunk * (size_t)M * 4);
    L.b = take((size_t)chunk * (size_t)M * 4);
    L.total = off;
    return L;
}

// f16: W holds binary16 values. radius >= 1; chunk >= 1 features per pass.
hipError_t launch_update(bool f16, void *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx,
                         int64_t N, int64_t nnz, const int32_t *bmu, int64_t radius, int64_t chunk,
                         const UpdateBuffers &ub, hipStream_t st);

}  // namespace som
