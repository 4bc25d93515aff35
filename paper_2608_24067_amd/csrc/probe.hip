// probe.hip -- a plain HBM read stream, the measured bandwidth denominator that the
// benchmark reports beside the published peak. Not part of the search: it lives in
// its own library (libsomprobe.so) and only the benchmark loads it.
//
// Every thread reads 16-byte vectors, eight in flight, over a grid-stride loop; the
// sum is written only if it equals a value no input of ones can produce, so the
// loads cannot be dropped and nothing is written in practice.

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_read_stream(const v4f *__restrict__ p, int64_t n, float *__restrict__ sink)
{
    const int64_t step = (int64_t)gridDim.x * 256;
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    float acc = 0.0f;
    for (; i + 7 * step < n; i += 8 * step) {
        v4f q[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) q[u] = p[i + u * step];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += q[u].x + q[u].y + q[u].z + q[u].w;
    }
    for (; i < n; i += step) acc += p[i].x + p[i].y + p[i].z + p[i].w;
    if (acc == -1.0f) sink[0] = acc;
}

}  // namespace

extern "C" {

// Reads the first `bytes` bytes (rounded down to 16) of the device buffer `buf` (16-byte
// aligned) once, on `stream`, with `blocks_per_cu` workgroups of 256 threads per compute
// unit (1 to 64). Returns 0, or a HIP error code. `sink`: one device float, written only
// for inputs that sum to -1.
int somprobe_read(const void *buf, size_t bytes, float *sink, int blocks_per_cu, void *stream)
{
    if (!buf || !sink || (reinterpret_cast<uintptr_t>(buf) & 15) || blocks_per_cu < 1 || blocks_per_cu > 64)
        return (int)hipErrorInvalidValue;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return (int)e;
    const int64_t n = (int64_t)(bytes / 16);
    hipLaunchKernelGGL(k_read_stream, dim3((unsigned)(cus * blocks_per_cu)), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const v4f *>(buf), n, sink);
    return (int)hipGetLastError();
}

}  // extern "C"
