// som_update.hip -- gfx950 kernels of the batch-SOM update (Algorithm 2, steps 8-9;
// factorised box-blur update section), for binary rows.
//
// After a search has given every sample its best unit, the update
//   1. scatters the batch onto the E x E lattice: den[i] = samples at unit i and,
//      feature by feature, num[v][i] = samples at unit i holding feature v (integer
//      atomics: exact and independent of their order);
//   2. converts both fields to fp32 and blurs them: three box passes along every
//      lattice row, then three along every lattice column, each a running window
//      sum over the clamped window (the first window summed in ascending order,
//      then per step the element entering added and the one leaving subtracted),
//      unnormalised -- the constant cancels in the quotient;
//   3. replaces every prototype by num / den (fp32 division), leaving a unit whose
//      blurred den is zero unchanged; an fp16 codebook receives the quotient
//      rounded once to binary16 at this final write.
// A lane owns one lattice line (row or column) of one field and runs its three
// passes sequentially, exactly in the order above, so the result is the same
// bits on every run. The row passes run on a transposed copy, so that in every
// pass neighbouring lanes read neighbouring addresses. Features are processed in chunks, so the workspace holds
// three fields of chunk * M values rather than V * M.

#include <climits>

#include "../../include/som.h"
#include "som_internal.h"

namespace som {
namespace {

// Samples per unit.
__global__ __launch_bounds__(256) void k_count_units(const int32_t *__restrict__ bmu, int64_t N, int64_t M,
                                                     int32_t *__restrict__ cnt)
{
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        const int32_t u = bmu[s];
        if (u >= 0 && u < M) atomicAdd(cnt + u, 1);
    }
}

// num[v - v0][unit of s] += 1 for every id v in [v0, v1) of every sample s.
__global__ __launch_bounds__(256) void k_count_features(const int32_t *__restrict__ row_ptr,
                                                        const int32_t *__restrict__ col_idx, int64_t N, int64_t nnz,
                                                        const int32_t *__restrict__ bmu, int64_t M, int32_t v0,
                                                        int32_t v1, int32_t *__restrict__ cnt)
{
    const int64_t base = row_ptr[0];
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        const int32_t u = bmu[s];
        if (u < 0 || u >= M) continue;
        int64_t rb = (int64_t)row_ptr[s] - base, re = (int64_t)row_ptr[s + 1] - base;
        rb = rb < 0 ? 0 : (rb > nnz ? nnz : rb);
        re = re < rb ? rb : (re > nnz ? nnz : re);
        for (int64_t p = rb; p < re; ++p) {
            const int32_t v = col_idx[base + p];
            if (v >= v0 && v < v1) atomicAdd(cnt + (int64_t)(v - v0) * M + u, 1);
        }
    }
}

// One running-sum box pass over a line of n values (stride apart), half-width r.
template <typename In>
__device__ __forceinline__ void box_pass(const In *in, float *out, int64_t n, int64_t stride, int64_t r)
{
    float s = 0.0f;
    for (int64_t j = 0; j <= r && j < n; ++j) s += (float)in[j * stride];
    out[0] = s;
    for (int64_t i = 1; i < n; ++i) {
        if (i + r < n) s += (float)in[(i + r) * stride];
        if (i - r - 1 >= 0) s -= (float)in[(i - r - 1) * stride];
        out[i * stride] = s;
    }
}

// Transpose of every field's E x E lattice, 64 x 64 tiles through LDS (padded
// against bank conflicts); the first use also converts the counts to fp32.
template <typename In>
__global__ __launch_bounds__(256) void k_transpose(const In *__restrict__ in, float *__restrict__ out, int64_t fields,
                                                   int64_t E)
{
    __shared__ float tile[64][65];
    const int64_t tiles_axis = (E + 63) / 64;
    const int64_t per_field = tiles_axis * tiles_axis;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4 threads
    for (int64_t t = blockIdx.x; t < fields * per_field; t += gridDim.x) {
        const int64_t f = t / per_field;
        const int64_t r0 = (t % per_field) / tiles_axis * 64, c0 = (t % per_field) % tiles_axis * 64;
        const In *src = in + f * E * E;
        float *dst = out + f * E * E;
        for (int y = ty; y < 64; y += 4)
            if (r0 + y < E && c0 + tx < E) tile[y][tx] = (float)src[(r0 + y) * E + c0 + tx];
        __syncthreads();
        for (int y = ty; y < 64; y += 4)
            if (c0 + y < E && r0 + tx < E) dst[(c0 + y) * E + r0 + tx] = tile[tx][y];
        __syncthreads();
    }
}

// Three passes along the lines that run down the lattice's second index, A -> B -> A
// -> B. One lane per (field, line): neighbouring lanes take neighbouring lines, so
// every step is one coalesced read. On a transposed field these are the row passes.
__global__ __launch_bounds__(256) void k_blur_down(float *__restrict__ a, float *__restrict__ b, int64_t fields,
                                                   int64_t E, int64_t r)
{
    const int64_t lines = fields * E;
    const int64_t M = E * E;
    for (int64_t l = (int64_t)blockIdx.x * 256 + threadIdx.x; l < lines; l += (int64_t)gridDim.x * 256) {
        const int64_t off = (l / E) * M + l % E;
        box_pass(a + off, b + off, E, E, r);
        box_pass(b + off, a + off, E, E, r);
        box_pass(a + off, b + off, E, E, r);
    }
}

// W[v0 + f][i] = num[f][i] / den[i] where den[i] > 0 (fp32; rounded once to binary16
// for an fp16 codebook), unchanged elsewhere.
template <typename E>
__global__ __launch_bounds__(256) void k_quotient(E *__restrict__ W, const float *__restrict__ num,
                                                  const float *__restrict__ den, int64_t fields, int64_t M, int64_t v0)
{
    const int64_t total = fields * M;
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < total; k += (int64_t)gridDim.x * 256) {
        const int64_t i = k % M;
        const float d = den[i];
        if (d > 0.0f) W[v0 * M + k] = (E)(num[k] / d);
    }
}

__global__ __launch_bounds__(256) void k_zero_i32(int32_t *__restrict__ p, int64_t n)
{
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256) p[k] = 0;
}

// Both fields' blur: counts (rows r, columns c) -> transposed fp32 (T[c][r]) -> row
// passes as passes down T -> transposed back -> column passes. Result in b.
void blur(const int32_t *cnt, float *a, float *b, int64_t fields, int64_t E, int64_t r, hipStream_t st);

unsigned grid_for(int64_t n)
{
    int64_t b = (n + 255) / 256;
    if (b < 1) b = 1;
    if (b > (1 << 20)) b = 1 << 20;
    return (unsigned)b;
}

void blur(const int32_t *cnt, float *a, float *b, int64_t fields, int64_t E, int64_t r, hipStream_t st)
{
    const int64_t tiles = fields * ((E + 63) / 64) * ((E + 63) / 64);
    const unsigned tg = (unsigned)(tiles < (1 << 20) ? tiles : (1 << 20));
    hipLaunchKernelGGL(k_transpose<int32_t>, dim3(tg), dim3(256), 0, st, cnt, a, fields, E);
    hipLaunchKernelGGL(k_blur_down, dim3(grid_for(fields * E)), dim3(256), 0, st, a, b, fields, E, r);
    hipLaunchKernelGGL(k_transpose<float>, dim3(tg), dim3(256), 0, st, b, a, fields, E);
    hipLaunchKernelGGL(k_blur_down, dim3(grid_for(fields * E)), dim3(256), 0, st, a, b, fields, E, r);
}

}  // namespace

hipError_t launch_update(bool f16, void *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx,
                         int64_t N, int64_t nnz, const int32_t *bmu, int64_t radius, int64_t chunk,
                         const UpdateBuffers &ub, hipStream_t st)
{
    const int64_t M = E * E;
    // den: counts, blur, kept in ub.den_b
    hipLaunchKernelGGL(k_zero_i32, dim3(grid_for(M)), dim3(256), 0, st, ub.den_cnt, M);
    hipLaunchKernelGGL(k_count_units, dim3(grid_for(N)), dim3(256), 0, st, bmu, N, M, ub.den_cnt);
    blur(ub.den_cnt, ub.den_a, ub.den_b, 1, E, radius, st);
    for (int64_t v0 = 0; v0 < V; v0 += chunk) {
        const int64_t f = V - v0 < chunk ? V - v0 : chunk;
        hipLaunchKernelGGL(k_zero_i32, dim3(grid_for(f * M)), dim3(256), 0, st, ub.cnt, f * M);
        hipLaunchKernelGGL(k_count_features, dim3(grid_for(N)), dim3(256), 0, st, row_ptr, col_idx, N, nnz, bmu, M,
                           (int32_t)v0, (int32_t)(v0 + f), ub.cnt);
        blur(ub.cnt, ub.a, ub.b, f, E, radius, st);
        if (f16)
            hipLaunchKernelGGL(k_quotient<_Float16>, dim3(grid_for(f * M)), dim3(256), 0, st,
                               static_cast<_Float16 *>(W), ub.b, ub.den_b, f, M, v0);
        else
            hipLaunchKernelGGL(k_quotient<float>, dim3(grid_for(f * M)), dim3(256), 0, st, static_cast<float *>(W),
                               ub.b, ub.den_b, f, M, v0);
    }
    return hipGetLastError();
}

}  // namespace som
