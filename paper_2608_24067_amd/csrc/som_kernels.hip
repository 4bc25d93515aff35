// som_kernels.hip -- gfx950 kernels of the sparse-binary BMU search.
//
// Method (SpMM-tile kernel section; Algorithm 2, steps 4-7): samples are
// grouped into tiles of TA consecutive rows; for each tile the distinct
// feature ids of its rows form the tile's union, each id carrying a TA-bit
// mask of the rows that hold it (k_plan). The sweep (k_sweep) gives each
// wave a strip of 256 neurons (4 per lane) of one tile: it streams the
// strip's segment of every union row once -- a coalesced 1 KiB read of the
// feature-major codebook W[v*M + i] -- and adds it into the register
// accumulators of every sample whose mask bit is set. A sample's dot product
// therefore is the fp32 sum of its own weights in ascending feature order,
// whatever TA is. The argmin is fused: each lane ranks its neurons by
// d = ||w||^2 - 2*dot in fp64, keeps the smallest 64-bit key per sample, and
// the wave and workgroup reduce the keys; one key per (sample, group of 1024
// neurons) leaves the kernel. k_finalize takes the smallest key per sample
// and recomputes the winner's full squared distance.
//
// Keys: the order-preserving image of the fp64 pattern of d (sign flipped
// for d >= 0, all bits flipped for d < 0), with its low 20 bits replaced by
// the neuron index. Comparing keys compares d (to 44 bits) and then the
// index, which gives the problem statement's lowest-index tie-break at every
// level of the reduction.

#include <climits>

#include "../../include/som.h"
#include "som_internal.h"

namespace som {
namespace {

typedef unsigned long long u64;

constexpr u64 kKeyNone = ~0ull;
constexpr u64 kIndexMask = (1ull << 20) - 1;

__device__ __forceinline__ u64 rank_key(double d, unsigned i)
{
    u64 b = (u64)__double_as_longlong(d);
    b = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
    return (b & ~kIndexMask) | (u64)i;
}

__device__ __forceinline__ u64 min_u64(u64 a, u64 b) { return b < a ? b : a; }

// ---- cross-lane helpers (DPP within a row of 16 lanes, readlane across rows)

// dpp_ctrl codes: quad_perm [1,0,3,2] = 0xB1 (lane ^ 1), quad_perm [2,3,0,1] = 0x4E
// (lane ^ 2), row_half_mirror = 0x141 (i <-> 7-i in each 8), row_mirror = 0x140
// (i <-> 15-i in each 16). Applied in this order every lane of a row ends with the
// row's minimum.
template <int CTRL>
__device__ __forceinline__ int dpp(int x)
{
    return __builtin_amdgcn_update_dpp(x, x, CTRL, 0xF, 0xF, false);
}

template <int CTRL>
__device__ __forceinline__ u64 dpp64(u64 x)
{
    const int lo = dpp<CTRL>((int)(unsigned)x);
    const int hi = dpp<CTRL>((int)(unsigned)(x >> 32));
    return ((u64)(unsigned)hi << 32) | (unsigned)lo;
}

__device__ __forceinline__ int wave_min_i32(int x)
{
    x = min(x, dpp<0xB1>(x));
    x = min(x, dpp<0x4E>(x));
    x = min(x, dpp<0x141>(x));
    x = min(x, dpp<0x140>(x));
    const int a = __builtin_amdgcn_readlane(x, 0), b = __builtin_amdgcn_readlane(x, 16);
    const int c = __builtin_amdgcn_readlane(x, 32), d = __builtin_amdgcn_readlane(x, 48);
    return min(min(a, b), min(c, d));
}

__device__ __forceinline__ u64 wave_min_u64(u64 x)
{
    x = min_u64(x, dpp64<0xB1>(x));
    x = min_u64(x, dpp64<0x4E>(x));
    x = min_u64(x, dpp64<0x141>(x));
    x = min_u64(x, dpp64<0x140>(x));
    u64 r = kKeyNone;
#pragma unroll
    for (int row = 0; row < 4; ++row) {
        const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)x, row * 16);
        const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(x >> 32), row * 16);
        r = min_u64(r, ((u64)hi << 32) | lo);
    }
    return r;
}

__device__ __forceinline__ int64_t clamp64(int64_t x, int64_t lo, int64_t hi) { return x < lo ? lo : (x > hi ? hi : x); }

// ----------------------------------------------------------------- norms

// n_i = sum_v W[v*M+i]^2: one thread per neuron, v ascending, fp64. The square of
// an fp32 value is exact in fp64, so fma(w, w, acc) equals acc + w*w.
__global__ __launch_bounds__(256) void k_norms(const float *__restrict__ W, int64_t V, int64_t M,
                                               double *__restrict__ norms)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= M) return;
    const float *p = W + i;
    double acc = 0.0;
    int64_t v = 0;
    for (; v + 8 <= V; v += 8) {
        float w[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) w[u] = __builtin_nontemporal_load(p + (v + u) * M);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const double x = (double)w[u];
            acc = fma(x, x, acc);
        }
    }
    for (; v < V; ++v) {
        const double x = (double)p[v * M];
        acc = fma(x, x, acc);
    }
    norms[i] = acc;
}

__global__ void k_clear_flags(uint32_t *flags) { flags[threadIdx.x] = 0u; }

// ------------------------------------------------------------------ plan

constexpr int kPlanWaves = 4;
constexpr int kPlanStage = 1024;  // ids of one tile staged in LDS per wave

// One wave per tile. Lane s < TA walks row t*TA+s; each step takes the smallest
// current id over the lanes (the next union element, ascending), the ballot of the
// lanes holding it (its sample mask), and advances those lanes: a TA-way merge of
// sorted lists. Offsets are clamped to [row_ptr[0], row_ptr[0]+nnz) and to the
// tile's own range, ids outside [0, V) are skipped, and a tile never writes more
// than its own CSR span of plan entries, so no input can drive an access out of
// bounds.
template <int TA>
__global__ __launch_bounds__(256) void k_plan(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                                              int64_t N, int64_t nnz, int32_t V, int64_t n_tiles,
                                              uint2 *__restrict__ plan, int2 *__restrict__ tiles,
                                              uint32_t *__restrict__ flags)
{
    __shared__ int32_t stage[kPlanWaves][kPlanStage];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t base = row_ptr[0];
    uint32_t bad = 0;

    for (int64_t t0 = (int64_t)blockIdx.x * kPlanWaves; t0 < n_tiles; t0 += (int64_t)gridDim.x * kPlanWaves) {
        const int64_t t = t0 + wv;
        const bool live = t < n_tiles;
        int64_t lo = 0, hi = 0, b = 0, e = 0;
        if (live) {
            const int64_t s0 = t * TA;
            const int64_t s1 = s0 + TA < N ? s0 + TA : N;
            lo = clamp64((int64_t)row_ptr[s0] - base, 0, nnz);
            hi = clamp64((int64_t)row_ptr[s1] - base, lo, nnz);
            if (lane < TA && s0 + lane < N) {
                const int64_t rb = (int64_t)row_ptr[s0 + lane] - base;
                const int64_t re = (int64_t)row_ptr[s0 + lane + 1] - base;
                if (re < rb || rb < lo || re > hi) bad |= SOM_FLAG_ROW_PTR;
                b = clamp64(rb, lo, hi);
                e = clamp64(re, b, hi);
            }
        }
        const bool staged = live && (hi - lo) <= kPlanStage;
        if (staged)
            for (int64_t q = lane; q < hi - lo; q += 64) stage[wv][q] = col_idx[base + lo + q];
        __syncthreads();
        if (live) {
            int64_t p = b;
            int cur = INT_MAX;
            // next valid id of this lane's row (INT_MAX when the row is done)
            auto fetch = [&]() {
                cur = INT_MAX;
                while (p < e) {
                    const int id = staged ? stage[wv][p - lo] : col_idx[base + p];
                    if (id >= 0 && id < V) {
                        cur = id;
                        break;
                    }
                    bad |= SOM_FLAG_ID_RANGE;
                    ++p;
                }
            };
            fetch();
            const int64_t cap = hi - lo;
            int64_t k = 0;
            while (true) {
                const int m = wave_min_i32(cur);
                if (m == INT_MAX) break;
                if (k >= cap) {  // only reachable with repeated or unsorted ids
                    bad |= SOM_FLAG_UNSORTED;
                    break;
                }
                const u64 mask = __ballot(cur == m);
                if (lane == 0) plan[lo + k] = make_uint2((unsigned)m, (unsigned)mask);
                ++k;
                if (cur == m) {
                    ++p;
                    fetch();
                    if (cur != INT_MAX && cur <= m) bad |= SOM_FLAG_UNSORTED;
                }
            }
            if (lane == 0) tiles[t] = make_int2((int)lo, (int)k);
        }
        __syncthreads();
    }
    if (bad) atomicOr(flags, bad);
}

// ----------------------------------------------------------------- sweep

// One workgroup = 4 waves = one tile x 1024 neurons (blockIdx.y selects the group
// of neurons, blockIdx.x strides over tiles, so the workgroups in flight share
// one group of codebook columns). Lane l of wave w owns neurons
// i0 = group*1024 + w*256 + 4*l .. i0+3. Lanes past M load a valid address and
// are never ranked.
// The plan is read defensively: offsets, counts and ids are clamped to the
// workspace and the codebook, so even a workspace the plan never wrote cannot
// drive an access out of bounds.
template <int TA, bool VEC>
__global__ __launch_bounds__(256) void k_sweep(const float *__restrict__ W, const double *__restrict__ norms,
                                               int64_t M, int64_t N, int64_t V, int64_t nnz,
                                               const uint2 *__restrict__ plan, const int2 *__restrict__ tiles,
                                               int64_t n_tiles, u64 *__restrict__ keys)
{
    __shared__ u64 red[kSweepWaves][TA];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t g = blockIdx.y;
    const int64_t i0 = g * kGroupNeurons + (int64_t)wv * kStripNeurons + (int64_t)lane * kNeuronsPerLane;

    // load columns: clamped so that every lane reads inside row v
    int64_t col[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) col[j] = VEC ? (i0 < M ? i0 : M - 4) + j : (i0 + j < M ? i0 + j : M - 1);
    double nrm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) nrm[j] = norms[col[j]];

    for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
        const int2 te = tiles[t];
        const int64_t off = clamp64(te.x, 0, nnz);
        const uint2 *ent = plan + off;
        const int cnt = (int)clamp64(te.y, 0, nnz - off);
        const unsigned vmax = (unsigned)(V - 1);

        float acc[TA][4];
#pragma unroll
        for (int s = 0; s < TA; ++s)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[s][j] = 0.0f;

        auto row_load = [&](unsigned id, float w[4]) {
            const float *r = W + (size_t)(id < vmax ? id : vmax) * (size_t)M;
            if (VEC) {
                const float4 q = *reinterpret_cast<const float4 *>(r + col[0]);
                w[0] = q.x;
                w[1] = q.y;
                w[2] = q.z;
                w[3] = q.w;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) w[j] = r[col[j]];
            }
        };
        auto row_add = [&](unsigned mask, const float w[4]) {
#pragma unroll
            for (int s = 0; s < TA; ++s) {
                if (mask & (1u << s)) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[s][j] += w[j];
                }
            }
        };

        int k = 0;
        for (; k + 4 <= cnt; k += 4) {
            uint2 en[4];
            float w[4][4];
#pragma unroll
            for (int u = 0; u < 4; ++u) en[u] = ent[k + u];
#pragma unroll
            for (int u = 0; u < 4; ++u) row_load(en[u].x, w[u]);
#pragma unroll
            for (int u = 0; u < 4; ++u) row_add(en[u].y, w[u]);
        }
        for (; k < cnt; ++k) {
            const uint2 en = ent[k];
            float w[4];
            row_load(en.x, w);
            row_add(en.y, w);
        }

        // fused argmin: d = ||w||^2 - 2*dot (fp64, one rounding), keyed
#pragma unroll
        for (int s = 0; s < TA; ++s) {
            u64 best = kKeyNone;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const double d = fma(-2.0, (double)acc[s][j], nrm[j]);
                const u64 key = (i0 + j < M) ? rank_key(d, (unsigned)(i0 + j)) : kKeyNone;
                best = min_u64(best, key);
            }
            best = wave_min_u64(best);
            if (lane == 0) red[wv][s] = best;
        }
        __syncthreads();
        if (threadIdx.x < TA) {
            const int s = threadIdx.x;
            u64 m = red[0][s];
#pragma unroll
            for (int w = 1; w < kSweepWaves; ++w) m = min_u64(m, red[w][s]);
            const int64_t row = t * TA + s;
            if (row < N) keys[g * N + row] = m;
        }
        __syncthreads();
    }
}

// -------------------------------------------------------------- finalize

// One thread per sample: smallest key over the groups, then the winner's distance
// from the sample's own ids, summed in the same order and precision as the sweep.
__global__ __launch_bounds__(256) void k_finalize(const float *__restrict__ W, const double *__restrict__ norms,
                                                  int32_t V, int64_t M, const int32_t *__restrict__ row_ptr,
                                                  const int32_t *__restrict__ col_idx, int64_t N, int64_t nnz,
                                                  const u64 *__restrict__ keys, int64_t n_groups,
                                                  int32_t *__restrict__ bmu, double *__restrict__ dist)
{
    const int64_t base = row_ptr[0];
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        u64 best = kKeyNone;
        for (int64_t g = 0; g < n_groups; ++g) best = min_u64(best, keys[g * N + s]);
        int64_t b = (int64_t)(best & kIndexMask);
        if (b >= M) b = M - 1;
        const int64_t rb = clamp64((int64_t)row_ptr[s] - base, 0, nnz);
        const int64_t re = clamp64((int64_t)row_ptr[s + 1] - base, rb, nnz);
        float dot = 0.0f;
        int cnt = 0;
        for (int64_t p = rb; p < re; ++p) {
            const int id = col_idx[base + p];
            if (id >= 0 && id < V) {
                dot += W[(size_t)id * (size_t)M + (size_t)b];
                ++cnt;
            }
        }
        bmu[s] = (int32_t)b;
        dist[s] = fma(-2.0, (double)dot, norms[b]) + (double)cnt;
    }
}

}  // namespace

// --------------------------------------------------------------- launchers

hipError_t launch_norms(const float *W, int64_t V, int64_t M, double *norms, hipStream_t st)
{
    const int64_t blocks = (M + 255) / 256;
    hipLaunchKernelGGL(k_norms, dim3((unsigned)blocks), dim3(256), 0, st, W, V, M, norms);
    return hipGetLastError();
}

hipError_t launch_clear_flags(uint32_t *flags, hipStream_t st)
{
    hipLaunchKernelGGL(k_clear_flags, dim3(1), dim3(64), 0, st, flags);
    return hipGetLastError();
}

hipError_t launch_plan(int ta, const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz, int64_t V,
                       uint2 *plan, int2 *tiles, uint32_t *flags, hipStream_t st)
{
    const int64_t n_tiles = (N + ta - 1) / ta;
    int64_t blocks = (n_tiles + kPlanWaves - 1) / kPlanWaves;
    if (blocks > (1 << 22)) blocks = 1 << 22;
    const dim3 grid((unsigned)blocks), block(256);
    switch (ta) {
    case 8: hipLaunchKernelGGL(k_plan<8>, grid, block, 0, st, row_ptr, col_idx, N, nnz, (int32_t)V, n_tiles, plan, tiles, flags); break;
    case 16: hipLaunchKernelGGL(k_plan<16>, grid, block, 0, st, row_ptr, col_idx, N, nnz, (int32_t)V, n_tiles, plan, tiles, flags); break;
    case 32: hipLaunchKernelGGL(k_plan<32>, grid, block, 0, st, row_ptr, col_idx, N, nnz, (int32_t)V, n_tiles, plan, tiles, flags); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int TA>
static void sweep_ta(bool vec, dim3 grid, hipStream_t st, const float *W, const double *norms, int64_t M, int64_t N,
                     int64_t V, int64_t nnz, const uint2 *plan, const int2 *tiles, int64_t n_tiles, u64 *keys)
{
    if (vec)
        hipLaunchKernelGGL((k_sweep<TA, true>), grid, dim3(256), 0, st, W, norms, M, N, V, nnz, plan, tiles, n_tiles,
                           keys);
    else
        hipLaunchKernelGGL((k_sweep<TA, false>), grid, dim3(256), 0, st, W, norms, M, N, V, nnz, plan, tiles,
                           n_tiles, keys);
}

hipError_t launch_sweep(int ta, const float *W, const double *norms, int64_t M, int64_t N, int64_t V, int64_t nnz,
                        const uint2 *plan, const int2 *tiles, unsigned long long *keys, int64_t n_groups,
                        hipStream_t st)
{
    const int64_t n_tiles = (N + ta - 1) / ta;
    int64_t gx = n_tiles > (1 << 22) ? (1 << 22) : n_tiles;
    const dim3 grid((unsigned)gx, (unsigned)n_groups);
    const bool vec = (M % 4 == 0) && ((reinterpret_cast<uintptr_t>(W) & 15) == 0);
    switch (ta) {
    case 8: sweep_ta<8>(vec, grid, st, W, norms, M, N, V, nnz, plan, tiles, n_tiles, keys); break;
    case 16: sweep_ta<16>(vec, grid, st, W, norms, M, N, V, nnz, plan, tiles, n_tiles, keys); break;
    case 32: sweep_ta<32>(vec, grid, st, W, norms, M, N, V, nnz, plan, tiles, n_tiles, keys); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_finalize(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                           const int32_t *col_idx, int64_t N, int64_t nnz, const unsigned long long *keys,
                           int64_t n_groups, int32_t *bmu, double *dist, hipStream_t st)
{
    int64_t blocks = (N + 255) / 256;
    if (blocks > (1 << 22)) blocks = 1 << 22;
    hipLaunchKernelGGL(k_finalize, dim3((unsigned)blocks), dim3(256), 0, st, W, norms, (int32_t)V, M, row_ptr,
                       col_idx, N, nnz, keys, n_groups, bmu, dist);
    return hipGetLastError();
}

}  // namespace som
