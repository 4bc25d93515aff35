// som_kernels.hip -- gfx950 kernels of the sparse-binary BMU search.
//
// Method (SpMM-tile kernel section; Algorithm 2, steps 4-7): samples are
// grouped into tiles of TA consecutive rows; for each tile the distinct
// feature ids of its rows form the tile's union, each id carrying a TA-bit
// mask of the rows that hold it (k_plan). In the sweep (k_sweep) a wave owns
// one tile and one strip of 64*NPL neurons (NPL per lane): it streams the
// strip's segment of every union row once -- a coalesced read of the
// feature-major codebook W[v*M + i] -- and adds it into the register
// accumulators of every sample whose mask bit is set. A sample's dot product
// therefore is the fp32 sum of its own weights in ascending feature order,
// whatever TA is. The argmin is fused: each lane ranks its neurons by
// d = ||w||^2 - 2*dot in fp64 and the wave reduces 64-bit keys per sample;
// one key per (sample, strip) leaves the kernel. k_finalize takes the
// smallest key per sample and recomputes the winner's full squared distance.
//
// A sweep workgroup takes groups of consecutive tiles of one strip (its four waves
// interleaved: wave w takes tiles w, w + 4, ...; up to 32 tiles per group), and
// blockIdx.y (the strip) is the slowest-varying dispatch index, so the workgroups
// in flight all read the same narrow column range of the codebook and its
// frequently used rows stay in L2.
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
typedef float v4f __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));

// Codebook element types: fp32, or IEEE binary16 storage (the paper's FP16 codebook,
// feature-major codebook section) widened to fp32 for the accumulation. Both
// conversions to fp32 and fp64 are exact.
//
// Elements per vector load in the sweep: 16 bytes, but no more than a lane's
// neurons (fp32: 4; fp16: 8, or 4 when a lane owns 4 neurons).
template <typename E, int NPL>
__host__ __device__ constexpr int group_elems()
{
    return (int)(16 / sizeof(E)) < NPL ? (int)(16 / sizeof(E)) : NPL;
}

// GRP consecutive elements at p (aligned to GRP * sizeof(E) bytes) as floats.
template <typename E, int GRP>
__device__ __forceinline__ void load_group(const E *p, float *w)
{
    if constexpr (sizeof(E) == 4) {
        static_assert(GRP == 4, "fp32 groups are 16 bytes");
        const v4f q = *reinterpret_cast<const v4f *>(p);
        w[0] = q.x;
        w[1] = q.y;
        w[2] = q.z;
        w[3] = q.w;
    } else if constexpr (GRP == 8) {
        const h8 q = *reinterpret_cast<const h8 *>(p);
#pragma unroll
        for (int k = 0; k < 8; ++k) w[k] = (float)q[k];
    } else {
        static_assert(GRP == 4, "fp16 groups are 8 or 16 bytes");
        const h4 q = *reinterpret_cast<const h4 *>(p);
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] = (float)q[k];
    }
}

constexpr u64 kKeyNone = ~0ull;
constexpr u64 kIndexMask = (1ull << 20) - 1;

__device__ __forceinline__ u64 rank_key(double d, unsigned i)
{
    u64 b = (u64)__double_as_longlong(d);
    b = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
    return (b & ~kIndexMask) | (u64)i;
}

__device__ __forceinline__ u64 min_u64(u64 a, u64 b) { return b < a ? b : a; }

__device__ __forceinline__ int64_t clamp64(int64_t x, int64_t lo, int64_t hi) { return x < lo ? lo : (x > hi ? hi : x); }

// The wave index as a scalar: threadIdx.x >> 6 is the same in every lane of a
// wave, but the compiler cannot prove it, and without this every value derived
// from it (tile index, plan entries, masks) would be treated as divergent.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// A compile-time bool carried as a type, for lambdas instantiated twice.
template <bool B>
struct StaticBool {
    static constexpr bool value = B;
};

// ---- cross-lane helpers (DPP within a row of 16 lanes, readlane across rows)

// dpp_ctrl codes: quad_perm [1,0,3,2] = 0xB1 (lane ^ 1), quad_perm [2,3,0,1] = 0x4E
// (lane ^ 2), row_half_mirror = 0x141 (i <-> 7-i in each 8), row_mirror = 0x140
// (i <-> 15-i in each 16). After the first k of these steps, every lane holds the
// minimum of its aligned group of 2, 4, 8 or 16 lanes.
template <int CTRL>
__device__ __forceinline__ int dpp(int x)
{
    return __builtin_amdgcn_update_dpp(x, x, CTRL, 0xF, 0xF, false);
}

// The same permutation for code where every lane of the wave is active: with
// bound_ctrl set the move can fold into the instruction that uses it.
template <int CTRL>
__device__ __forceinline__ int dpp_all(int x)
{
    return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, true);
}

template <int CTRL>
__device__ __forceinline__ u64 dpp64(u64 x)
{
    const int lo = dpp<CTRL>((int)(unsigned)x);
    const int hi = dpp<CTRL>((int)(unsigned)(x >> 32));
    return ((u64)(unsigned)hi << 32) | (unsigned)lo;
}

// Minimum over each aligned group of G lanes (G = 2, 4, 8, 16 or 32), in every lane of the
// group; every lane of the wave active.
template <int G>
__device__ __forceinline__ int group_min_i32(int x)
{
    x = min(x, dpp_all<0xB1>(x));
    if (G >= 4) x = min(x, dpp_all<0x4E>(x));
    if (G >= 8) x = min(x, dpp_all<0x141>(x));
    if (G >= 16) x = min(x, dpp_all<0x140>(x));
    if (G >= 32) x = min(x, __shfl_xor(x, 16));
    return x;
}

// Minimum over the whole wave, as a scalar.
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

// Order-preserving integer image of a float (signed comparison of images = comparison
// of finite values; -0 sorts just below +0, a NaN beyond the infinity of its sign),
// and its inverse. Integer minima fold into DPP-modified instructions, float ones
// would need a canonicalising move per step.
__device__ __forceinline__ int ord_f32(float f)
{
    const int b = __float_as_int(f);
    return b ^ ((b >> 31) & 0x7FFFFFFF);
}
__device__ __forceinline__ float from_ord_f32(int k) { return __int_as_float(k ^ ((k >> 31) & 0x7FFFFFFF)); }

// Minimum of a float over the whole wave (every lane active), as a scalar, through
// the integer images.
__device__ __forceinline__ float wave_min_f32(float x)
{
    int k = ord_f32(x);
    k = min(k, dpp_all<0xB1>(k));
    k = min(k, dpp_all<0x4E>(k));
    k = min(k, dpp_all<0x141>(k));
    k = min(k, dpp_all<0x140>(k));
    int r = __builtin_amdgcn_readlane(k, 0);
#pragma unroll
    for (int row = 1; row < 4; ++row) r = min(r, __builtin_amdgcn_readlane(k, row * 16));
    return from_ord_f32(r);
}

// Maximum of a float over the whole wave, as a scalar (NaN lanes are ignored unless
// every lane is NaN).

__device__ __forceinline__ float wave_max_f32(float x)
{
    x = fmaxf(x, __int_as_float(dpp<0xB1>(__float_as_int(x))));
    x = fmaxf(x, __int_as_float(dpp<0x4E>(__float_as_int(x))));
    x = fmaxf(x, __int_as_float(dpp<0x141>(__float_as_int(x))));
    x = fmaxf(x, __int_as_float(dpp<0x140>(__float_as_int(x))));
    float r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
#pragma unroll
    for (int row = 1; row < 4; ++row) r = fmaxf(r, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), row * 16)));
    return r;
}

__device__ __forceinline__ u64 readlane_u64(u64 x, int l)
{
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)x, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(x >> 32), l);
    return ((u64)hi << 32) | lo;
}

// The two smallest of the wave's values, each lane contributing the pair
// (a1 <= a2): merging (a1, a2) with (b1, b2) keeps min(a1, b1) and
// min(max(a1, b1), min(a2, b2)). On the integer images, every lane active; results
// are scalars.
__device__ __forceinline__ void min2_merge(int &a1, int &a2, int b1, int b2)
{
    const int lo = min(a1, b1);
    a2 = min(max(a1, b1), min(a2, b2));
    a1 = lo;
}

template <int CTRL>
__device__ __forceinline__ void min2_step(int &a1, int &a2)
{
    min2_merge(a1, a2, dpp_all<CTRL>(a1), dpp_all<CTRL>(a2));
}

__device__ __forceinline__ void wave_min2_f32(float x1, float x2, float &r1, float &r2)
{
    int a1 = ord_f32(x1), a2 = ord_f32(x2);
    min2_step<0xB1>(a1, a2);
    min2_step<0x4E>(a1, a2);
    min2_step<0x141>(a1, a2);
    min2_step<0x140>(a1, a2);
    int s1 = __builtin_amdgcn_readlane(a1, 0), s2 = __builtin_amdgcn_readlane(a2, 0);
#pragma unroll
    for (int row = 1; row < 4; ++row)
        min2_merge(s1, s2, __builtin_amdgcn_readlane(a1, row * 16), __builtin_amdgcn_readlane(a2, row * 16));
    r1 = from_ord_f32(s1);
    r2 = from_ord_f32(s2);
}

// ----------------------------------------------------------------- norms

// n_i = sum_v W[v*M+i]^2: one thread per neuron, v ascending, fp64. The square of
// an fp32 (or fp16) value is exact in fp64, so fma(w, w, acc) equals acc + w*w.
// One wave per workgroup, so a small map (M = 4096: 64 waves) still spreads over
// 64 compute units, and kNormLoads rows in flight per wave: the sums are sequential,
// the loads are not.
constexpr int kNormLoads = 32;

template <typename E>
__global__ __launch_bounds__(64) void k_norms(const E *__restrict__ W, int64_t V, int64_t M,
                                              double *__restrict__ norms)
{
    const int64_t i = (int64_t)blockIdx.x * 64 + threadIdx.x;
    if (i >= M) return;
    const E *p = W + i;
    double acc = 0.0;
    int64_t v = 0;
    for (; v + kNormLoads <= V; v += kNormLoads) {
        float w[kNormLoads];
#pragma unroll
        for (int u = 0; u < kNormLoads; ++u) w[u] = (float)__builtin_nontemporal_load(p + (v + u) * M);
#pragma unroll
        for (int u = 0; u < kNormLoads; ++u) {
            const double x = (double)w[u];
            acc = fma(x, x, acc);
        }
    }
    for (; v < V; ++v) {
        const double x = (double)(float)p[v * M];
        acc = fma(x, x, acc);
    }
    norms[i] = acc;
}

__global__ void k_clear_flags(uint32_t *flags) { flags[threadIdx.x] = 0u; }

// ----------------------------------------------------------------- order

// Sample order. The post-submission section's tuning groups samples so that a
// tile's rows share features. Here the samples of a batch are bucketed by their
// least frequent feature in that batch: rows that share a rare feature land in
// the same or neighbouring tiles, which run close together in time, so a rare
// codebook row is re-read while still in L2. A sample's result does not depend on where it
// sits (its sum order is fixed by its own features), so the permutation never
// shows in the output. The permuted batch is written to the workspace as a CSR
// of its own (prp, pci); k_unpermute moves the results back to their samples.

constexpr int kLdsHistMax = 32768;          // features whose counts fit the LDS histogram
constexpr int64_t kFreqSample = 1ll << 25;  // ids counted: the ordering needs only a rough rarity rank

__global__ __launch_bounds__(256) void k_fill_u32(uint32_t *__restrict__ p, int64_t n, uint32_t v)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = v;
}

__global__ __launch_bounds__(256) void k_fill_u64(u64 *__restrict__ p, int64_t n, u64 v)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = v;
}

// freq[v] = occurrences of feature v among the batch's first kFreqSample ids (all of
// them for smaller batches; ids outside [0, V) skipped). Each workgroup counts a
// contiguous chunk in LDS, then adds its non-zero counts to the global histogram.
__global__ __launch_bounds__(256) void k_freq(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                                              int64_t nnz, int32_t V, uint32_t *__restrict__ freq)
{
    __shared__ uint32_t h[kLdsHistMax];
    const int64_t base = row_ptr[0];
    const bool lds = V <= kLdsHistMax;
    if (lds)
        for (int v = threadIdx.x; v < V; v += 256) h[v] = 0u;
    __syncthreads();
    const int64_t chunk = (nnz + gridDim.x - 1) / gridDim.x;
    const int64_t p0 = (int64_t)blockIdx.x * chunk;
    const int64_t p1 = p0 + chunk < nnz ? p0 + chunk : nnz;
    for (int64_t p = p0 + threadIdx.x; p < p1; p += 256) {
        const int id = col_idx[base + p];
        if (id >= 0 && id < V) {
            if (lds) atomicAdd(&h[id], 1u);
            else atomicAdd(&freq[id], 1u);
        }
    }
    __syncthreads();
    if (lds)
        for (int v = threadIdx.x; v < V; v += 256)
            if (h[v]) atomicAdd(&freq[v], h[v]);
}

// Clamped id range of row s (relative to row_ptr[0]); empty if row_ptr decreases.
__device__ __forceinline__ void row_range(const int32_t *row_ptr, int64_t base, int64_t nnz, int64_t s, int64_t &rb,
                                          int64_t &re, uint32_t &bad)
{
    const int64_t a = (int64_t)row_ptr[s] - base, b = (int64_t)row_ptr[s + 1] - base;
    if (b < a || a < 0 || b > nnz) bad |= SOM_FLAG_ROW_PTR;
    rb = clamp64(a, 0, nnz);
    re = b < a ? rb : clamp64(b, rb, nnz);
}

// skey[s] = the sample's least frequent valid feature (ties: the larger id), V if it
// has none; bucket[key] += (1 << 32) | row length: samples counted in the high
// half, ids in the low half of one 64-bit word.
__global__ __launch_bounds__(256) void k_rarest(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                                                int64_t N, int64_t nnz, int32_t V, const uint32_t *__restrict__ freq,
                                                int32_t *__restrict__ skey, u64 *__restrict__ bucket,
                                                uint32_t *__restrict__ flags)
{
    // the four lanes of a quad share a row (lane q of the quad takes ids q, q + 4, ...)
    const int64_t base = row_ptr[0];
    const int sub = threadIdx.x & 3;
    uint32_t bad = 0;
    for (int64_t s = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2); s < N; s += (int64_t)gridDim.x * 64) {
        int64_t rb, re;
        row_range(row_ptr, base, nnz, s, rb, re, bad);
        u64 best = kKeyNone;  // (frequency, V-1-id): smallest frequency, then largest id
        // three of the lane's ids, then their counts, per step: a row of up to 12 ids is one
        // round trip of dependent loads instead of three
        for (int64_t p = rb + sub; p < re; p += 12) {
            int id[3];
#pragma unroll
            for (int j = 0; j < 3; ++j) id[j] = p + 4 * j < re ? col_idx[base + p + 4 * j] : -1;
            unsigned f[3];
#pragma unroll
            for (int j = 0; j < 3; ++j) f[j] = id[j] >= 0 && id[j] < V ? freq[id[j]] : 0u;
#pragma unroll
            for (int j = 0; j < 3; ++j)
                if (id[j] >= 0 && id[j] < V) best = min_u64(best, ((u64)f[j] << 32) | (unsigned)(V - 1 - id[j]));
        }
        // the quad is active or idle as a whole (one row), so the swaps read its own lanes
        best = min_u64(best, dpp64<0xB1>(best));
        best = min_u64(best, dpp64<0x4E>(best));
        if (sub == 0) {
            const int key = best == kKeyNone ? V : (int)(V - 1 - (int)(unsigned)(best & 0xFFFFFFFFull));
            skey[s] = key;
            atomicAdd(&bucket[key], (1ull << 32) | (u64)(re - rb));
        }
    }
    if (bad) atomicOr(flags, bad);
}

// One workgroup: exclusive scan of the nb packed bucket counts into packed starting
// offsets (sample offset << 32 | id offset). prp[N] = total ids (capped at nnz).
__global__ __launch_bounds__(1024) void k_bucket_scan(u64 *__restrict__ bucket, int64_t nb, int64_t nnz,
                                                      int32_t *__restrict__ prp_end)
{
    __shared__ int64_t ss[1024], si[1024];
    const int t = threadIdx.x;
    const int64_t per = (nb + 1023) / 1024;
    const int64_t b0 = t * per < nb ? t * per : nb;
    const int64_t b1 = b0 + per < nb ? b0 + per : nb;
    int64_t ns = 0, ni = 0;
    for (int64_t b = b0; b < b1; ++b) {
        ns += (int64_t)(bucket[b] >> 32);
        ni += (int64_t)(bucket[b] & 0xFFFFFFFFull);
    }
    ss[t] = ns;
    si[t] = ni;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {  // inclusive Hillis-Steele scan
        const int64_t a = t >= d ? ss[t - d] : 0, c = t >= d ? si[t - d] : 0;
        __syncthreads();
        ss[t] += a;
        si[t] += c;
        __syncthreads();
    }
    int64_t os = ss[t] - ns, oi = si[t] - ni;  // exclusive
    for (int64_t b = b0; b < b1; ++b) {
        const u64 c = bucket[b];
        bucket[b] = ((u64)os << 32) | (u64)(oi & 0xFFFFFFFFll);
        os += (int64_t)(c >> 32);
        oi += (int64_t)(c & 0xFFFFFFFFull);
    }
    if (t == 1023) *prp_end = (int32_t)(si[1023] < nnz ? si[1023] : nnz);
}

// Each sample takes the next (position, id offset) of its bucket with one atomic and
// copies its ids (and values, for real-valued rows) there: sample s sits at position
// inv[s] of the permuted batch, its ids from pci[prp[inv[s]]] on. A quad of
// lanes shares a row: its first lane takes the atomic, the quad copies every
// fourth id, so the reads of row_ptr and col_idx run in batch order and only the
// writes scatter, as whole rows. Positions past N and id offsets past nnz (only
// reachable with invalid row pointers) are dropped or clamped.
constexpr int kPlaceLanes = 4;

__global__ __launch_bounds__(256) void k_place(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                                               int64_t N, int64_t nnz, const int32_t *__restrict__ skey,
                                               u64 *__restrict__ bucket, int32_t *__restrict__ inv,
                                               int32_t *__restrict__ prp, int32_t *__restrict__ pci,
                                               const float *__restrict__ values, float *__restrict__ pvals)
{
    const int64_t base = row_ptr[0];
    const int sub = threadIdx.x % kPlaceLanes;
    constexpr int64_t per_block = 256 / kPlaceLanes;
    uint32_t bad = 0;
    for (int64_t s = (int64_t)blockIdx.x * per_block + threadIdx.x / kPlaceLanes; s < N;
         s += (int64_t)gridDim.x * per_block) {
        int64_t rb, re;
        row_range(row_ptr, base, nnz, s, rb, re, bad);
        u64 old = 0;
        if (sub == 0) old = atomicAdd(&bucket[skey[s]], (1ull << 32) | (u64)(re - rb));
        // the quad is active or idle as a whole (one row): its lanes read lane 0's word
        old = dpp64<0x00>(old);
        const int64_t ps = (int64_t)(old >> 32), pi = (int64_t)(old & 0xFFFFFFFFull);
        if (sub == 0) inv[s] = ps < N ? (int32_t)ps : -1;
        if (ps >= N) continue;
        const int64_t dst = pi < nnz ? pi : nnz;
        if (sub == 0) prp[ps] = (int32_t)dst;
        const int64_t n = re - rb < nnz - dst ? re - rb : nnz - dst;
        const int32_t *src = col_idx + base + rb;
        int32_t *out = pci + dst;
        for (int64_t q = sub; q < n; q += kPlaceLanes) out[q] = src[q];
        if (values) {
            const float *vs = values + base + rb;
            float *vo = pvals + dst;
            for (int64_t q = sub; q < n; q += kPlaceLanes) vo[q] = vs[q];
        }
    }
}

// ------------------------------------------------------------------ plan

constexpr int kPlanWaves = 4;
constexpr int kPlanStage = 2048;  // ids staged in LDS per wave

// A wave plans 64/TA consecutive tiles at once (TA = 2 ... 32): lane l works on row s = l % TA of
// tile l / TA. Each step takes, per tile, the smallest current id over its TA
// lanes (the next element of the union, ascending), the ballot of the lanes
// holding it (its sample mask), and advances those lanes: a TA-way merge of
// sorted lists per lane group. Offsets are clamped to [row_ptr[0], row_ptr[0]+nnz)
// and to each tile's own range, ids outside [0, V) are skipped, and a tile never
// writes more entries than its own CSR span, so no input can drive an access out
// of bounds.
//
// Real-valued rows (REAL, values given): every union entry also gets the TA values of
// its samples (vals[entry*TA + s], written for the samples whose mask bit is set;
// the other slots are never read), and every row the fp64 sum of its squared
// values in its own order (xsq, by batch position), which is ||x||^2.
template <int TA, bool REAL>
__global__ __launch_bounds__(256) void k_plan(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                                              int64_t N, int64_t nnz, int32_t V, int64_t n_tiles,
                                              uint2 *__restrict__ plan, int2 *__restrict__ tiles,
                                              uint32_t *__restrict__ flags, const float *__restrict__ values,
                                              float *__restrict__ vals, double *__restrict__ xsq)
{
    constexpr int G = 64 / TA;  // tiles per wave
    __shared__ int32_t stage[kPlanWaves][kPlanStage];
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    const int grp = lane / TA;
    const int sl = lane % TA;
    const int64_t base = row_ptr[0];
    uint32_t bad = 0;

    for (int64_t tb = (int64_t)blockIdx.x * kPlanWaves * G; tb < n_tiles; tb += (int64_t)gridDim.x * kPlanWaves * G) {
        const int64_t tw = tb + (int64_t)wv * G;  // first tile of this wave
        const int64_t t = tw + grp;               // this lane's tile
        const bool live = t < n_tiles;
        // the wave's CSR span, for staging
        int64_t wlo = 0, whi = 0;
        if (tw < n_tiles) {
            const int64_t te = tw + G < n_tiles ? tw + G : n_tiles;
            wlo = clamp64((int64_t)row_ptr[tw * TA] - base, 0, nnz);
            whi = clamp64((int64_t)row_ptr[te * TA < N ? te * TA : N] - base, wlo, nnz);
        }
        int64_t lo = 0, hi = 0, b = 0, e = 0;
        if (live) {
            const int64_t s0 = t * TA;
            const int64_t s1 = s0 + TA < N ? s0 + TA : N;
            lo = clamp64((int64_t)row_ptr[s0] - base, wlo, whi);
            hi = clamp64((int64_t)row_ptr[s1] - base, lo, whi);
            if (s0 + sl < N) {
                const int64_t rb = (int64_t)row_ptr[s0 + sl] - base;
                const int64_t re = (int64_t)row_ptr[s0 + sl + 1] - base;
                if (re < rb || rb < lo || re > hi) bad |= SOM_FLAG_ROW_PTR;
                b = clamp64(rb, lo, hi);
                e = clamp64(re, b, hi);
            }
        }
        const bool staged = (whi - wlo) <= kPlanStage;  // wave-uniform
        if (staged)
            for (int64_t q = lane; q < whi - wlo; q += 64) stage[wv][q] = col_idx[base + wlo + q];
        __syncthreads();

        // positions in 32 bits: every offset lies in [0, nnz] and nnz < 2^31
        const int32_t *ids = col_idx + base;
        const float *vsrc = REAL ? values + base : nullptr;
        int p = (int)b;
        const int pe = (int)e, plo = (int)lo, pwlo = (int)wlo;
        int cur = INT_MAX;
        float curv = 0.0f;
        double sq = 0.0;
        int k = 0;  // union entries written for this lane's tile (equal across its group)
        // The merge, in two copies: ids read from the LDS stage or from global memory.
        // (One copy with a select between the two pointers becomes a flat load that
        // waits on both memory counters at every step.)
        auto merge = [&](auto from_stage) {
            constexpr bool STAGED = decltype(from_stage)::value;
            auto id_at = [&](int q) {
                if constexpr (STAGED)
                    return stage[wv][q - pwlo];
                else
                    return ids[q];
            };
            // next valid id of this lane's row (INT_MAX once the row is done), with its value;
            // ids outside [0, V) (invalid input) are skipped on a path of their own
            auto fetch = [&]() {
                cur = INT_MAX;
                if (p >= pe) return;
                int id = id_at(p);
                if (id < 0 || id >= V) {
                    for (;;) {
                        bad |= SOM_FLAG_ID_RANGE;
                        if (++p >= pe) return;
                        id = id_at(p);
                        if (id >= 0 && id < V) break;
                    }
                }
                cur = id;
                if constexpr (REAL) {
                    curv = vsrc[p];
                    sq = fma((double)curv, (double)curv, sq);
                }
            };
            fetch();
            // Every step consumes at least one id of the group, so a tile takes at most as many
            // steps as its span holds ids; only lanes whose ranges overlap (row pointers that
            // decrease, flagged above) take more, and their surplus entries are dropped.
            const int cap = (int)(hi - lo);
            while (true) {
                const int m = group_min_i32<TA>(cur);
                if (__ballot(m != INT_MAX) == 0) break;
                const u64 bal = __ballot(m != INT_MAX && cur == m);
                const unsigned mask =
                    (unsigned)((bal >> (grp * TA)) & (TA == 32 ? 0xFFFFFFFFull : ((1ull << TA) - 1)));
                if (m != INT_MAX) {
                    if (k < cap) {
                        if (sl == 0) plan[plo + k] = make_uint2((unsigned)m, mask);
                        if (REAL && cur == m) vals[(int64_t)(plo + k) * TA + sl] = curv;
                    }
                    ++k;
                    if (cur == m) {
                        ++p;
                        fetch();
                        if (cur != INT_MAX && cur <= m) bad |= SOM_FLAG_UNSORTED;
                    }
                }
            }
        };
        if (staged)
            merge(StaticBool<true>{});
        else
            merge(StaticBool<false>{});
        if (live && sl == 0) tiles[t] = make_int2((int)lo, k < (int)(hi - lo) ? k : (int)(hi - lo));
        if (REAL && live && t * TA + sl < N) xsq[t * TA + sl] = sq;
        __syncthreads();
    }
    if (bad) atomicOr(flags, bad);
}

// ----------------------------------------------------------------- sweep

// Workgroup = 4 waves x one strip (blockIdx.y) of 64*NPL neurons, over groups of
// group_tiles consecutive tiles (a multiple of 4; groups blockIdx.x, blockIdx.x +
// gridDim.x, ...); each lane owns NPL neurons, in groups of G (four fp32 values, or
// min(8, NPL) fp16 ones; see loc below). VEC: M is a multiple of G and W aligned to a
// group's bytes, so each group is one aligned vector load (16 bytes; 8 for fp16 at four
// neurons per lane).
// The plan is read defensively (offsets, counts and ids clamped to the workspace
// and the codebook), so even a workspace the plan never wrote cannot drive an
// access out of bounds.
//
// TOP2: each (sample, strip) also gets its second-smallest key and that neuron's dot
// product (keys2, dots2), for the two best units of the fused sweep.
//
// REAL: real-valued rows (the Discussion's gather-multiply variant). The plan holds
// each union entry's TA sample values (vals); a set mask bit adds value * weight
// (one fused multiply-add, fp32) instead of the weight, still in ascending feature
// order per sample.
template <typename E, int TA, int NPL, int U, bool VEC, bool TOP2, bool REAL>
__global__ __launch_bounds__(256) void k_sweep(const E *__restrict__ W, const double *__restrict__ norms,
                                               int64_t M, int64_t N, int64_t V, int64_t nnz,
                                               const uint2 *__restrict__ plan, const int2 *__restrict__ tiles,
                                               int64_t n_tiles, u64 *__restrict__ keys, float *__restrict__ dots,
                                               u64 *__restrict__ keys2, float *__restrict__ dots2,
                                               const float *__restrict__ vals, int64_t group_tiles)
{
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    const int64_t strip = blockIdx.y;
    // M <= 2^20: neuron indices and byte offsets within a row fit in 32 bits.
    const int Mi = (int)M;
    const int base = (int)strip * (64 * NPL);  // first neuron of the strip
    // Element j of lane l is neuron base + loc(j), loc(j) = (j/G)*64G + G*l + j%G with
    // G = group_elems (4 for fp32): each group of G is one vector load, and the 64
    // lanes' loads of a group cover one contiguous stretch of the row (1 KiB for fp32
    // and for fp16 at 8 neurons per lane).
    constexpr int G = group_elems<E, NPL>();
    const int lg = lane * G;
    // a lane's part of one codebook row, as stored
    struct Seg {
        typedef E vec __attribute__((ext_vector_type(G)));
        union {
            vec v[NPL / G];
            E e[NPL];
        };
    };
    auto loc = [&](int j) { return (j / G) * (64 * G) + lg + (j % G); };

    // fp64 norms, +inf past M (those neurons then never pass the candidate test
    // below); nmax = the largest fp32 norm of the strip.
    double nrm[NPL];
    float nmax_l = 0.0f;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int i = base + loc(j);
        nrm[j] = i < Mi ? norms[i] : __builtin_inf();
        if (i < Mi) nmax_l = fmaxf(nmax_l, (float)nrm[j]);
    }
    const float nmax = wave_max_f32(nmax_l);
    const unsigned vmax = (unsigned)(V - 1);

    // Tiles wv, wv + 4, ... of the workgroup's groups. The next tile's header (its plan
    // offset and union size, and the next tile's offset that bounds it) and its first
    // U plan entries are fetched while the current tile is still being worked on, so
    // no scalar-load latency sits between two tiles.
    int64_t gbeg = (int64_t)blockIdx.x * group_tiles;  // first tile of the current group
    int64_t t = gbeg + wv;
    if (t >= n_tiles) return;  // wave-uniform; this kernel has no barriers
    // the wave's tile after t (n_tiles when there is none), and its group's first tile
    auto next_tile = [&](int64_t &gb) {
        int64_t n = t + 4;
        gb = gbeg;
        if (n >= gbeg + group_tiles) {
            gb = gbeg + (int64_t)gridDim.x * group_tiles;
            n = gb + wv;
        }
        return n < n_tiles ? n : n_tiles;
    };
    // header of tile tt from its table entry and the next tile's offset (nnz past the
    // last tile): a tile's union never reaches the next tile's span
    auto header = [&](int2 te, int next_off, int64_t &off_o, int &cnt_o) {
        off_o = clamp64(te.x, 0, nnz);
        cnt_o = (int)clamp64(te.y, 0, clamp64(next_off, off_o, nnz) - off_o);
    };
    auto next_offset = [&](int64_t tt) { return tt + 1 < n_tiles ? tiles[tt + 1].x : (int)nnz; };
    int64_t off;
    int cnt;
    header(tiles[t], next_offset(t), off, cnt);
    uint2 nx[U];
    if (cnt >= U) {
#pragma unroll
        for (int u = 0; u < U; ++u) nx[u] = plan[off + u];
    }
    for (;;) {
        const uint2 *ent = plan + off;
        int64_t gbeg_n;
        const int64_t tn = next_tile(gbeg_n);

        float acc[TA][NPL];
#pragma unroll
        for (int s = 0; s < TA; ++s)
#pragma unroll
            for (int j = 0; j < NPL; ++j) acc[s][j] = 0.0f;

        // A row segment is held as loaded (fp16 stays packed, half the registers) and
        // widened when it is added. Lanes whose group lies past M (last strip only)
        // re-read the row's last group; those neurons are never ranked.
        auto row_load = [&](unsigned id, Seg &seg) {
            // 32 x 32-bit product: ids < 2^31 and M <= 2^20
            const E *r = W + (uint64_t)(id < vmax ? id : vmax) * (uint64_t)(unsigned)Mi;
            if constexpr (VEC) {
#pragma unroll
                for (int q = 0; q < NPL / G; ++q) {
                    const int g = base + loc(q * G);
                    seg.v[q] = *reinterpret_cast<const typename Seg::vec *>(r + (g < Mi ? g : Mi - G));
                }
            } else {
#pragma unroll
                for (int j = 0; j < NPL; ++j) {
                    const int g = base + loc(j);
                    seg.e[j] = r[g < Mi ? g : Mi - 1];
                }
            }
        };
        // The mask is wave-uniform: each bit is a scalar branch, tested four bits at a
        // time first (an entry usually has one or two bits set). The empty volatile
        // asm keeps the compiler from turning the branch into unconditional adds
        // and selects.
        auto each_sample = [&](unsigned mask, auto &&body) {
#pragma unroll
            for (int s0 = 0; s0 < TA; s0 += 4) {
                if (mask & (0xFu << s0)) {
#pragma unroll
                    for (int s = s0; s < s0 + 4; ++s) {
                        if (mask & (1u << s)) {
                            body(s);
                            asm volatile("");
                        }
                    }
                }
            }
        };
        // xv: the entry's TA sample values (REAL only; scalar registers)
        auto row_add = [&](unsigned mask, const Seg &seg, const float *xv) {
            if constexpr (sizeof(E) == 2 && VEC) {
                // Packed fp16: each update is one mixed-precision FMA with h read as a
                // half straight from the loaded dword (exact widening, one rounding):
                // acc + h * 1.0, or acc + h * x for real values -- the same result as
                // widening first.
                const unsigned *dw = reinterpret_cast<const unsigned *>(&seg.v[0]);
                each_sample(mask, [&](int s) {
#pragma unroll
                        for (int d = 0; d < NPL / 2; ++d) {
                            if constexpr (REAL) {
                                asm("v_fma_mix_f32 %0, %1, %2, %0 op_sel_hi:[1,0,0]"
                                    : "+v"(acc[s][2 * d])
                                    : "v"(dw[d]), "s"(xv[s]));
                                asm("v_fma_mix_f32 %0, %1, %2, %0 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
                                    : "+v"(acc[s][2 * d + 1])
                                    : "v"(dw[d]), "s"(xv[s]));
                            } else {
                                asm("v_fma_mix_f32 %0, %1, 1.0, %0 op_sel_hi:[1,0,0]"
                                    : "+v"(acc[s][2 * d])
                                    : "v"(dw[d]));
                                asm("v_fma_mix_f32 %0, %1, 1.0, %0 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
                                    : "+v"(acc[s][2 * d + 1])
                                    : "v"(dw[d]));
                            }
                        }
                });
            } else {
                float w[NPL];
#pragma unroll
                for (int j = 0; j < NPL; ++j) {
                    if constexpr (VEC)
                        w[j] = (float)seg.v[j / G][j % G];
                    else
                        w[j] = (float)seg.e[j];
                }
                each_sample(mask, [&](int s) {
#pragma unroll
                    for (int j = 0; j < NPL; ++j) {
                        if constexpr (REAL)
                            acc[s][j] = fmaf(xv[s], w[j], acc[s][j]);
                        else
                            acc[s][j] += w[j];
                    }
                });
            }
        };
        // the TA sample values of plan entry q (REAL only)
        auto entry_values = [&](int64_t q, float *xv) {
            if constexpr (REAL) {
                const float *src = vals + (off + q) * TA;
#pragma unroll
                for (int s = 0; s < TA; ++s) xv[s] = src[s];
            }
        };

        // U rows in flight; the next U plan entries are fetched (scalar loads) while
        // the current rows are loaded and added.
        int k = 0;
        for (; k + U <= cnt; k += U) {
            uint2 en[U];
#pragma unroll
            for (int u = 0; u < U; ++u) en[u] = nx[u];
            if (k + 2 * U <= cnt) {
#pragma unroll
                for (int u = 0; u < U; ++u) nx[u] = ent[k + U + u];
            }
            Seg seg[U];
#pragma unroll
            for (int u = 0; u < U; ++u) row_load(en[u].x, seg[u]);
            float xv[U][TA];
#pragma unroll
            for (int u = 0; u < U; ++u) entry_values(k + u, xv[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) row_add(en[u].y, seg[u], xv[u]);
        }
        for (; k < cnt; ++k) {
            const uint2 en = ent[k];
            Seg seg;
            row_load(en.x, seg);
            float xv[TA];
            entry_values(k, xv);
            row_add(en.y, seg, xv);
        }
        // The next tile's table entries are read now, its first plan entries halfway
        // through this tile's epilogue; both are in flight while the epilogue runs.
        int2 te_n = make_int2(0, 0);
        int next_n = 0;
        if (tn < n_tiles) {
            te_n = tiles[tn];
            next_n = next_offset(tn);
        }
        int64_t off_n = 0;
        int cnt_n = 0;

        // Fused argmin, exact, in two stages. Stage 1 ranks the strip in fp32:
        // da = fl32(fl32(n_i) - 2*dot) differs from the fp64 distance d = fl64(n_i - 2*dot)
        // by at most 2^-24 (n_i + |da|) + 2^-53 |d|. So the neuron with the smallest key
        // (smallest d to the key's 44 bits, then lowest index) has
        // da <= min(da) + 2^-20 (nmax + |min(da)| + 1), which leaves room for both
        // errors and for the key's 2^-32 relative truncation. Stage 2 forms the fp64
        // distance and key of those candidates only -- usually one neuron in the strip
        // -- so the smallest key is the one a full fp64 pass would find. A non-finite
        // threshold (overflowing norms or sums) sends every neuron to stage 2.
        float nf[NPL];  // converted once per tile (the asm keeps it out of the main loop's registers)
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            double x = nrm[j];
            asm volatile("" : "+v"(x));
            nf[j] = (float)x;
        }
        u64 mine = kKeyNone, mine2 = kKeyNone;
        float mine_dot = 0.0f, mine_dot2 = 0.0f;
#pragma unroll
        for (int s = 0; s < TA; ++s) {
            if (s == TA / 2 && tn < n_tiles) {
                header(te_n, next_n, off_n, cnt_n);
                if (cnt_n >= U) {
#pragma unroll
                    for (int u = 0; u < U; ++u) nx[u] = plan[off_n + u];
                }
            }
            float da[NPL];
            if constexpr (!TOP2) {
                float lmin = __builtin_inff();
#pragma unroll
                for (int j = 0; j < NPL; ++j) {
                    da[j] = fmaf(-2.0f, acc[s][j], nf[j]);
                    lmin = fminf(lmin, da[j]);
                }
                const float wmin = wave_min_f32(lmin);
                const float thr = wmin + 0x1p-20f * (nmax + fabsf(wmin) + 1.0f);
                const bool every = !(fabsf(thr) <= __FLT_MAX__);
                // Keys carry the neuron's index within the strip; the strip's first
                // neuron is added once the strip's smallest key is known.
                u64 best = kKeyNone;
                float bdot = 0.0f;
                auto visit = [&](int j, bool cand) {
                    const double d = fma(-2.0, (double)acc[s][j], nrm[j]);
                    const bool take = cand && base + loc(j) < Mi;
                    const u64 key = take ? rank_key(d, (unsigned)loc(j)) : kKeyNone;
                    if (key < best) {
                        best = key;
                        bdot = acc[s][j];
                    }
                };
                // The common case tests each neuron group with one compare and skips it
                // when no lane holds a candidate; a non-finite bound takes every neuron.
                if (!every) {
#pragma unroll
                    for (int j = 0; j < NPL; ++j)
                        if (__builtin_amdgcn_ballot_w64(da[j] <= thr)) visit(j, da[j] <= thr);
                } else {
#pragma unroll
                    for (int j = 0; j < NPL; ++j) visit(j, true);
                }
                // Lane s keeps sample s's smallest key over the strip and the dot
                // product of the lane that owns it (index within the strip mod 64G =
                // G * lane + j % G).
                const u64 holders = __builtin_amdgcn_ballot_w64(best != kKeyNone);
                int owner;
                if (__popcll(holders) == 1) {
                    owner = __builtin_ctzll(holders);
                    best = readlane_u64(best, owner);
                } else {
                    best = wave_min_u64(best);
                    owner = (int)((best & (64 * G - 1)) / G);
                }
                const float dot = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bdot), owner));
                if (best != kKeyNone) best += (u64)base;
                if (lane == s) {
                    mine = best;
                    mine_dot = dot;
                }
            } else {
                // Stage 1 with the two smallest approximate distances: the neurons of
                // the two smallest keys have da <= (second smallest da) + eps.
                float m1 = __builtin_inff(), m2 = __builtin_inff();
#pragma unroll
                for (int j = 0; j < NPL; ++j) {
                    da[j] = fmaf(-2.0f, acc[s][j], nf[j]);
                    m2 = fminf(m2, fmaxf(m1, da[j]));
                    m1 = fminf(m1, da[j]);
                }
                float w1, w2;
                wave_min2_f32(m1, m2, w1, w2);
                const float thr = w2 + 0x1p-20f * (nmax + fabsf(w1) + fabsf(w2) + 1.0f);
                const bool every = !(fabsf(thr) <= __FLT_MAX__);
                u64 k1 = kKeyNone, k2 = kKeyNone;
                float q1 = 0.0f, q2 = 0.0f;
                auto visit = [&](int j, bool cand) {
                    const double d = fma(-2.0, (double)acc[s][j], nrm[j]);
                    const bool take = cand && base + loc(j) < Mi;
                    const u64 key = take ? rank_key(d, (unsigned)loc(j)) : kKeyNone;
                    if (key < k1) {
                        k2 = k1;
                        q2 = q1;
                        k1 = key;
                        q1 = acc[s][j];
                    } else if (key < k2) {
                        k2 = key;
                        q2 = acc[s][j];
                    }
                };
                if (!every) {
#pragma unroll
                    for (int j = 0; j < NPL; ++j)
                        if (__builtin_amdgcn_ballot_w64(da[j] <= thr)) visit(j, da[j] <= thr);
                } else {
#pragma unroll
                    for (int j = 0; j < NPL; ++j) visit(j, true);
                }
                // The two smallest keys of the wave (keys are distinct: each holds its
                // neuron index), with the dot products of their neurons.
                u64 K1, K2;
                float D1, D2;
                const u64 h1 = __builtin_amdgcn_ballot_w64(k1 != kKeyNone);
                const u64 h2 = __builtin_amdgcn_ballot_w64(k2 != kKeyNone);
                const int n1 = __popcll(h1), n2 = __popcll(h2);
                if (n1 + n2 <= 2) {
                    // at most two keys in the wave: read them directly
                    const int la = n1 ? __builtin_ctzll(h1) : 0;
                    u64 A = n1 ? readlane_u64(k1, la) : kKeyNone;
                    float DA = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q1), la));
                    u64 B = kKeyNone;
                    float DB = 0.0f;
                    if (n1 == 2) {
                        const int lb = __builtin_ctzll(h1 & (h1 - 1));
                        B = readlane_u64(k1, lb);
                        DB = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q1), lb));
                    } else if (n2 == 1) {
                        B = readlane_u64(k2, la);
                        DB = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q2), la));
                    }
                    const bool swap = B < A;
                    K1 = swap ? B : A;
                    D1 = swap ? DB : DA;
                    K2 = swap ? A : B;
                    D2 = swap ? DA : DB;
                } else {
                    K1 = wave_min_u64(k1);
                    const int o1 = __builtin_ctzll(__builtin_amdgcn_ballot_w64(k1 == K1));
                    D1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q1), o1));
                    // the owner of K1 offers its second key, every other lane its first
                    const u64 nxt = lane == o1 ? k2 : k1;
                    const float nq = lane == o1 ? q2 : q1;
                    K2 = wave_min_u64(nxt);
                    const u64 h = __builtin_amdgcn_ballot_w64(nxt == K2 && K2 != kKeyNone);
                    const int o2 = h ? __builtin_ctzll(h) : 0;
                    D2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(nq), o2));
                }
                if (K1 != kKeyNone) K1 += (u64)base;
                if (K2 != kKeyNone) K2 += (u64)base;
                if (lane == s) {
                    mine = K1;
                    mine_dot = D1;
                    mine2 = K2;
                    mine_dot2 = D2;
                }
            }
        }
        const int64_t row = t * TA + lane;
        if (lane < TA && row < N) {
            keys[strip * N + row] = mine;
            dots[strip * N + row] = mine_dot;
            if constexpr (TOP2) {
                keys2[strip * N + row] = mine2;
                dots2[strip * N + row] = mine_dot2;
            }
        }
        if (tn >= n_tiles) break;
        t = tn;
        gbeg = gbeg_n;
        off = off_n;
        cnt = cnt_n;
    }
}

// -------------------------------------------------------------- finalize

// One thread per position k of the (possibly permuted) batch: smallest key over the
// strips; the winner's dot product comes from the sweep (the same fp32 sum of the
// row's weights in ascending feature order), so the full squared distance is
// (||w||^2 - 2*dot) + ||x||^2, with ||x||^2 = nnz for binary rows and xsq[k] from the
// plan for real-valued ones. Results are written by position (k_unpermute then moves
// them to their samples when the batch was regrouped): every write coalesced.
// Where a finalize kernel puts a position's result: the caller's arrays (positions are
// samples) or, for a regrouped batch, one staged record per position.
struct FinalOut {
    int32_t *bmu;
    double *dist;
    Staged *rec;  // non-null: staged
    __device__ void put(int64_t k, int32_t b, double d) const
    {
        if (rec) {
            rec[k] = Staged{d, b, 0};
        } else {
            bmu[k] = b;
            dist[k] = d;
        }
    }
};

constexpr int kFinalizeBatch = 8;   // strips whose keys one lane loads at once
constexpr int kFinalize2Batch = 4;  // the same for the two-best search (four words per strip)

__global__ __launch_bounds__(256) void k_finalize(const double *__restrict__ norms, int64_t M,
                                                  const int32_t *__restrict__ row_ptr, int64_t N, int64_t nnz,
                                                  const double *__restrict__ xsq,
                                                  const u64 *__restrict__ keys,
                                                  const float *__restrict__ dots, int64_t n_strips,
                                                  FinalOut out)
{
    const int64_t base = row_ptr[0];
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < N; k += (int64_t)gridDim.x * 256) {
        u64 best = kKeyNone;
        int64_t gb = 0;
        for (int64_t g0 = 0; g0 < n_strips; g0 += kFinalizeBatch) {
            // a batch of strips' keys loaded before any is compared
            u64 kk[kFinalizeBatch];
#pragma unroll
            for (int j = 0; j < kFinalizeBatch; ++j) kk[j] = g0 + j < n_strips ? keys[(g0 + j) * N + k] : kKeyNone;
#pragma unroll
            for (int j = 0; j < kFinalizeBatch; ++j)
                if (kk[j] < best) {
                    best = kk[j];
                    gb = g0 + j;
                }
        }
        int64_t b = (int64_t)(best & kIndexMask);
        if (b >= M) b = M - 1;
        const int64_t rb = clamp64((int64_t)row_ptr[k] - base, 0, nnz);
        const int64_t re = clamp64((int64_t)row_ptr[k + 1] - base, rb, nnz);
        out.put(k, (int32_t)b, fma(-2.0, (double)dots[gb * N + k], norms[b]) + (xsq ? xsq[k] : (double)(re - rb)));
    }
}

// Two best units: the two smallest of the 2 * n_strips keys of each sample (each
// strip's two smallest), with their dot products from the sweep. Without a second
// unit (M == 1) bmu2 = -1 and dist2 = +inf.
__global__ __launch_bounds__(256) void k_finalize2(const double *__restrict__ norms, int64_t M,
                                                   const int32_t *__restrict__ row_ptr, int64_t N, int64_t nnz,
                                                   const double *__restrict__ xsq,
                                                   const u64 *__restrict__ keys,
                                                   const float *__restrict__ dots, const u64 *__restrict__ keys2,
                                                   const float *__restrict__ dots2, int64_t n_strips,
                                                   FinalOut out, FinalOut out2)
{
    const int64_t base = row_ptr[0];
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < N; k += (int64_t)gridDim.x * 256) {
        u64 b1 = kKeyNone, b2 = kKeyNone;
        float q1 = 0.0f, q2 = 0.0f;
        auto offer = [&](u64 key, float q) {
            if (key < b1) {
                b2 = b1;
                q2 = q1;
                b1 = key;
                q1 = q;
            } else if (key < b2) {
                b2 = key;
                q2 = q;
            }
        };
        for (int64_t g0 = 0; g0 < n_strips; g0 += kFinalize2Batch) {
            // a batch of strips' candidates loaded before any is offered, offered in strip order
            u64 k1[kFinalize2Batch], k2[kFinalize2Batch];
            float d1[kFinalize2Batch], d2[kFinalize2Batch];
#pragma unroll
            for (int j = 0; j < kFinalize2Batch; ++j) {
                const bool in = g0 + j < n_strips;
                const int64_t at = (g0 + j) * N + k;
                k1[j] = in ? keys[at] : kKeyNone;
                d1[j] = in ? dots[at] : 0.0f;
                k2[j] = in ? keys2[at] : kKeyNone;
                d2[j] = in ? dots2[at] : 0.0f;
            }
#pragma unroll
            for (int j = 0; j < kFinalize2Batch; ++j) {
                offer(k1[j], d1[j]);
                offer(k2[j], d2[j]);
            }
        }
        const int64_t rb = clamp64((int64_t)row_ptr[k] - base, 0, nnz);
        const int64_t re = clamp64((int64_t)row_ptr[k + 1] - base, rb, nnz);
        const double len = xsq ? xsq[k] : (double)(re - rb);
        int64_t i1 = (int64_t)(b1 & kIndexMask);
        if (i1 >= M) i1 = M - 1;
        out.put(k, (int32_t)i1, fma(-2.0, (double)q1, norms[i1]) + len);
        if (b2 == kKeyNone) {
            out2.put(k, -1, __builtin_inf());
        } else {
            int64_t i2 = (int64_t)(b2 & kIndexMask);
            if (i2 >= M) i2 = M - 1;
            out2.put(k, (int32_t)i2, fma(-2.0, (double)q2, norms[i2]) + len);
        }
    }
}

// Results of a regrouped batch back to input order: sample s takes what position inv[s]
// got (bmu2/dist2 too when given). A sample never placed (inv[s] = -1, invalid row
// pointers only) is left untouched. Reads gather, writes run in sample order.
__global__ __launch_bounds__(256) void k_unpermute(const int32_t *__restrict__ inv, int64_t N,
                                                   const Staged *__restrict__ res, const Staged *__restrict__ res2,
                                                   int32_t *__restrict__ bmu,
                                                   double *__restrict__ dist, int32_t *__restrict__ bmu2,
                                                   double *__restrict__ dist2)
{
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        const int64_t k = inv[s];
        if (k < 0 || k >= N) continue;
        const Staged r = res[k];
        bmu[s] = r.b;
        dist[s] = r.d;
        if (bmu2) {
            const Staged r2 = res2[k];
            bmu2[s] = r2.b;
            dist2[s] = r2.d;
        }
    }
}

}  // namespace

// --------------------------------------------------------------- launchers

hipError_t launch_norms(const float *W, int64_t V, int64_t M, double *norms, hipStream_t st)
{
    const int64_t blocks = (M + 63) / 64;
    hipLaunchKernelGGL(k_norms<float>, dim3((unsigned)blocks), dim3(64), 0, st, W, V, M, norms);
    return hipGetLastError();
}

hipError_t launch_norms_f16(const uint16_t *W, int64_t V, int64_t M, double *norms, hipStream_t st)
{
    const int64_t blocks = (M + 63) / 64;
    hipLaunchKernelGGL(k_norms<_Float16>, dim3((unsigned)blocks), dim3(64), 0, st,
                       reinterpret_cast<const _Float16 *>(W), V, M, norms);
    return hipGetLastError();
}

hipError_t launch_clear_flags(uint32_t *flags, hipStream_t st)
{
    hipLaunchKernelGGL(k_clear_flags, dim3(1), dim3(64), 0, st, flags);
    return hipGetLastError();
}

hipError_t launch_plan(int ta, const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N,
                       int64_t nnz, int64_t V, uint2 *plan, int2 *tiles, float *vals, double *xsq, uint32_t *flags,
                       hipStream_t st)
{
    const int64_t nt = n_tiles(N, ta);
    const int64_t per_block = (int64_t)kPlanWaves * (64 / ta);
    int64_t blocks = (nt + per_block - 1) / per_block;
    if (blocks > (1 << 22)) blocks = 1 << 22;
    const dim3 grid((unsigned)blocks), block(256);
    const int32_t v = (int32_t)V;
    if (values) {  // real-valued rows: tiles of 8 only
        if (ta != 8) return hipErrorInvalidValue;
        hipLaunchKernelGGL((k_plan<8, true>), grid, block, 0, st, row_ptr, col_idx, N, nnz, v, nt, plan, tiles, flags,
                           values, vals, xsq);
        return hipGetLastError();
    }
    switch (ta) {
    case 8:
        hipLaunchKernelGGL((k_plan<8, false>), grid, block, 0, st, row_ptr, col_idx, N, nnz, v, nt, plan, tiles, flags,
                           nullptr, nullptr, nullptr);
        break;
    case 16:
        hipLaunchKernelGGL((k_plan<16, false>), grid, block, 0, st, row_ptr, col_idx, N, nnz, v, nt, plan, tiles,
                           flags, nullptr, nullptr, nullptr);
        break;
    case 32:
        hipLaunchKernelGGL((k_plan<32, false>), grid, block, 0, st, row_ptr, col_idx, N, nnz, v, nt, plan, tiles,
                           flags, nullptr, nullptr, nullptr);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename E, int TA, int NPL, bool TOP2, bool REAL>
static void sweep_ta(bool vec, dim3 grid, int64_t group_tiles, hipStream_t st, const E *W, const double *norms,
                     int64_t M, int64_t N, int64_t V, int64_t nnz, const uint2 *plan, const int2 *tiles, int64_t nt,
                     const SweepOut &o, const float *vals)
{
    // Packed fp16 rows take half the registers: eight rows in flight still fit 128 VGPRs
    // (six for real-valued rows, whose per-entry values take scalar registers).
    constexpr int UV = (sizeof(E) == 2 && NPL == 8) ? (REAL ? 6 : 8) : 4;
    if (vec)
        hipLaunchKernelGGL((k_sweep<E, TA, NPL, UV, true, TOP2, REAL>), grid, dim3(256), 0, st, W, norms, M, N, V, nnz,
                           plan, tiles, nt, o.keys, o.dots, o.keys2, o.dots2, vals, group_tiles);
    else
        hipLaunchKernelGGL((k_sweep<E, TA, NPL, 4, false, TOP2, REAL>), grid, dim3(256), 0, st, W, norms, M, N, V, nnz,
                           plan, tiles, nt, o.keys, o.dots, o.keys2, o.dots2, vals, group_tiles);
}

// Consecutive tiles per sweep workgroup. Longer groups let a wave keep its strip's
// norms over several tiles and keep the tiles in flight a compact stretch of the
// (regrouped) batch, but a strip must still span many rounds of resident
// workgroups, or the chip works on two strips at once and their rows compete for
// L2: up to 32 tiles, and at least 16,384 groups per strip where there are enough.
static int64_t sweep_group_tiles(int64_t nt)
{
    int64_t g = nt / 16384 / 4 * 4;
    return g < 4 ? 4 : (g > 32 ? 32 : g);
}

// Vector loads need M to be a multiple of the group and W aligned to the group's bytes.
template <typename E, int NPL>
static bool vector_loads(const E *W, int64_t M)
{
    constexpr int G = group_elems<E, NPL>();
    return M % G == 0 && (reinterpret_cast<uintptr_t>(W) % (G * sizeof(E))) == 0;
}

template <typename E, bool TOP2>
static hipError_t sweep_any(int ta, const E *W, const double *norms, int64_t M, int64_t N, int64_t V, int64_t nnz,
                            const uint2 *plan, const int2 *tiles, const float *vals, const SweepOut &o,
                            hipStream_t st)
{
    const int64_t nt = n_tiles(N, ta);
    const int64_t gt = sweep_group_tiles(nt);
    int64_t gx = (nt + gt - 1) / gt;
    if (gx > (1 << 20)) gx = 1 << 20;
    const dim3 grid((unsigned)gx, (unsigned)n_strips(M, ta));
    if (vals) {  // real-valued rows: tiles of 8 only (8 values per plan entry in scalar registers)
        if (ta != 8) return hipErrorInvalidValue;
        sweep_ta<E, 8, 8, TOP2, true>(vector_loads<E, 8>(W, M), grid, gt, st, W, norms, M, N, V, nnz, plan, tiles,
                                      nt, o, vals);
        return hipGetLastError();
    }
    switch (ta) {
    case 8:
        sweep_ta<E, 8, 8, TOP2, false>(vector_loads<E, 8>(W, M), grid, gt, st, W, norms, M, N, V, nnz, plan, tiles,
                                       nt, o, nullptr);
        break;
    case 16:
        sweep_ta<E, 16, 4, TOP2, false>(vector_loads<E, 4>(W, M), grid, gt, st, W, norms, M, N, V, nnz, plan, tiles,
                                        nt, o, nullptr);
        break;
    case 32:
        sweep_ta<E, 32, 4, TOP2, false>(vector_loads<E, 4>(W, M), grid, gt, st, W, norms, M, N, V, nnz, plan, tiles,
                                        nt, o, nullptr);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_sweep(int ta, bool f16, bool top2, const void *W, const double *norms, int64_t M, int64_t N,
                        int64_t V, int64_t nnz, const uint2 *plan, const int2 *tiles, const float *vals,
                        const SweepOut &o, hipStream_t st)
{
    if (f16) {
        const _Float16 *w = static_cast<const _Float16 *>(W);
        return top2 ? sweep_any<_Float16, true>(ta, w, norms, M, N, V, nnz, plan, tiles, vals, o, st)
                    : sweep_any<_Float16, false>(ta, w, norms, M, N, V, nnz, plan, tiles, vals, o, st);
    }
    const float *w = static_cast<const float *>(W);
    return top2 ? sweep_any<float, true>(ta, w, norms, M, N, V, nnz, plan, tiles, vals, o, st)
                : sweep_any<float, false>(ta, w, norms, M, N, V, nnz, plan, tiles, vals, o, st);
}

hipError_t launch_finalize(int ta, const double *norms, int64_t M, const int32_t *row_ptr, int64_t N, int64_t nnz,
                           const OrderBuffers *ob, const double *xsq, const SweepOut &o, int32_t *bmu, double *dist,
                           int32_t *bmu2, double *dist2, hipStream_t st)
{
    int64_t blocks = (N + 255) / 256;
    if (blocks > (1 << 22)) blocks = 1 << 22;
    // a regrouped batch is finalized by position into the workspace first
    const FinalOut o1{bmu, dist, ob ? ob->res : nullptr}, o2{bmu2, dist2, ob ? ob->res2 : nullptr};
    if (bmu2)
        hipLaunchKernelGGL(k_finalize2, dim3((unsigned)blocks), dim3(256), 0, st, norms, M, row_ptr, N, nnz, xsq,
                           o.keys, o.dots, o.keys2, o.dots2, n_strips(M, ta), o1, o2);
    else
        hipLaunchKernelGGL(k_finalize, dim3((unsigned)blocks), dim3(256), 0, st, norms, M, row_ptr, N, nnz, xsq,
                           o.keys, o.dots, n_strips(M, ta), o1);
    if (ob)
        hipLaunchKernelGGL(k_unpermute, dim3((unsigned)blocks), dim3(256), 0, st, ob->inv, N, ob->res,
                           bmu2 ? ob->res2 : nullptr, bmu, dist, bmu2, dist2);
    return hipGetLastError();
}

hipError_t launch_order(const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N, int64_t nnz,
                        int64_t V, const OrderBuffers &ob, uint32_t *flags, hipStream_t st)
{
    const int64_t nb = V + 1;  // one bucket per feature, one for rows without a valid feature
    int64_t fb = (nb + 255) / 256;
    if (fb > 4096) fb = 4096;
    hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)fb), dim3(256), 0, st, ob.freq, nb, 0u);
    hipLaunchKernelGGL(k_fill_u64, dim3((unsigned)fb), dim3(256), 0, st, ob.bucket, nb, 0ull);
    // enough workgroups to fill the chip, each with a large chunk of ids for its LDS histogram
    const int64_t counted = nnz < kFreqSample ? nnz : kFreqSample;
    int64_t hb = (counted + 65535) / 65536;
    if (hb < 1) hb = 1;
    if (hb > 1024) hb = 1024;
    hipLaunchKernelGGL(k_freq, dim3((unsigned)hb), dim3(256), 0, st, row_ptr, col_idx, counted, (int32_t)V, ob.freq);
    int64_t qb = (N + 63) / 64;  // a row per quad of lanes
    if (qb > (1 << 22)) qb = 1 << 22;
    hipLaunchKernelGGL(k_rarest, dim3((unsigned)qb), dim3(256), 0, st, row_ptr, col_idx, N, nnz, (int32_t)V, ob.freq,
                       ob.skey, ob.bucket, flags);
    hipLaunchKernelGGL(k_bucket_scan, dim3(1), dim3(1024), 0, st, ob.bucket, nb, nnz, ob.prp + N);
    int64_t pb = (N + 256 / kPlaceLanes - 1) / (256 / kPlaceLanes);
    if (pb > (1 << 22)) pb = 1 << 22;
    hipLaunchKernelGGL(k_place, dim3((unsigned)pb), dim3(256), 0, st, row_ptr, col_idx, N, nnz, ob.skey, ob.bucket,
                       ob.inv, ob.prp, ob.pci, values, values ? ob.pvals : nullptr);
    return hipGetLastError();
}

}  // namespace som
