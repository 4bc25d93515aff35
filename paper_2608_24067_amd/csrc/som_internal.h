// som_internal.h -- shared between the C-ABI layer and the kernels of libsom.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace som {

// Neurons per lane in the sweep (one 16-byte load per codebook row).
constexpr int kNeuronsPerLane = 4;
// Waves per sweep workgroup; the waves of a workgroup take consecutive strips of one tile.
constexpr int kSweepWaves = 4;
// Neurons one sweep wave covers, and one workgroup (a "group" of the partial-key array).
constexpr int kStripNeurons = 64 * kNeuronsPerLane;
constexpr int kGroupNeurons = kSweepWaves * kStripNeurons;
// Smallest tile the plan supports: the plan's tile table is sized for it.
constexpr int kMinTileSamples = 8;
constexpr int kDefaultTileSamples = 16;

// Workspace carve-up (offsets in bytes from the workspace base; every section 256-byte aligned).
struct Layout {
    size_t plan;     // uint2 [nnz]: (feature id, sample mask) of every tile's union, tile t at its CSR offset
    size_t tiles;    // int2 [ceil(N / kMinTileSamples)]: (plan offset, union size) per tile
    size_t keys;     // uint64 [n_groups * N]: per-group partial argmin keys, group-major
    size_t flags;    // uint32 [64]: input flags
    size_t total;
    int64_t n_groups;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline Layout layout_for(int64_t N, int64_t M, int64_t nnz)
{
    Layout L;
    L.n_groups = (M + kGroupNeurons - 1) / kGroupNeurons;
    const int64_t max_tiles = (N + kMinTileSamples - 1) / kMinTileSamples;
    size_t off = 0;
    L.plan = off;
    off += align256((size_t)nnz * 8);
    L.tiles = off;
    off += align256((size_t)max_tiles * 8);
    L.keys = off;
    off += align256((size_t)L.n_groups * (size_t)N * 8);
    L.flags = off;
    off += 256;
    L.total = off;
    return L;
}

// Kernel launchers (som_kernels.hip). Each returns the launch's hipError_t.
hipError_t launch_norms(const float *W, int64_t V, int64_t M, double *norms, hipStream_t st);
hipError_t launch_clear_flags(uint32_t *flags, hipStream_t st);
hipError_t launch_plan(int ta, const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz, int64_t V,
                       uint2 *plan, int2 *tiles, uint32_t *flags, hipStream_t st);
hipError_t launch_sweep(int ta, const float *W, const double *norms, int64_t M, int64_t N, int64_t V, int64_t nnz,
                        const uint2 *plan, const int2 *tiles, unsigned long long *keys, int64_t n_groups,
                        hipStream_t st);
hipError_t launch_finalize(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                           const int32_t *col_idx, int64_t N, int64_t nnz, const unsigned long long *keys,
                           int64_t n_groups, int32_t *bmu, double *dist, hipStream_t st);

}  // namespace som
