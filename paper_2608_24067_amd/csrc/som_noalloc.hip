// som_noalloc.hip -- som_bmu_search_noalloc: the single-best BMU search with its scratch
// space in a file-scope device array instead of a caller's workspace, for callers that
// cannot allocate device memory (code under stream capture, tight serving loops,
// harnesses that forbid allocation). It runs exactly the kernels of som_bmu_search.
//
// The array is part of the library's code object: every GPU the library runs on holds
// its own copy, at its own address, until the process ends. Its device address is taken
// once per device, with that device current, on the first call there; host code never
// passes the array's name to a kernel or a copy, only that address.

#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/som.h"
#include "som_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[SOM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void *g_scratch[kMaxDevices];
hipError_t g_status[kMaxDevices];
std::once_flag g_once[kMaxDevices];

}  // namespace

extern "C" som_status som_bmu_search_noalloc(const float *W, const double *norms, int64_t V, int64_t M,
                                             const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz,
                                             int32_t *bmu, double *dist, const som_bmu_config *config, void *stream)
{
    const char *who = "som_bmu_search_noalloc";
    const size_t need = som_bmu_workspace_bytes(N, M, V, nnz, config);
    if (need == 0)
        return som::set_error(SOM_ERR_INVALID_ARG, "%s: sizes or config out of range (N=%lld M=%lld V=%lld nnz=%lld)",
                              who, (long long)N, (long long)M, (long long)V, (long long)nnz);
    if (need > (size_t)SOM_NOALLOC_SCRATCH_BYTES)
        return som::set_error(SOM_ERR_WORKSPACE,
                              "%s: this search needs %zu bytes of scratch, the library's array holds %zu; "
                              "use som_bmu_search with a workspace of som_bmu_workspace_bytes",
                              who, need, (size_t)SOM_NOALLOC_SCRATCH_BYTES);
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return som::set_error(SOM_ERR_HIP, "%s: hipGetDevice: %s", who, hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return som::set_error(SOM_ERR_INVALID_ARG, "%s: device %d is beyond the %d this entry point serves", who, dev,
                              kMaxDevices);
    std::call_once(g_once[dev], [dev] { g_status[dev] = hipGetSymbolAddress(&g_scratch[dev], HIP_SYMBOL(scratch)); });
    if (g_status[dev] != hipSuccess)
        return som::set_error(SOM_ERR_HIP, "%s: hipGetSymbolAddress on device %d: %s", who, dev,
                              hipGetErrorString(g_status[dev]));
    return som_bmu_search(W, norms, V, M, row_ptr, col_idx, N, nnz, bmu, dist, g_scratch[dev],
                          (size_t)SOM_NOALLOC_SCRATCH_BYTES, config, stream);
}
