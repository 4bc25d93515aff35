// som_device.h -- device helpers shared by the kernels of libsom.so (som_kernels.hip,
// som_sweep.hip): element loads, the 64-bit argmin keys, clamping, DPP and lane
// reductions.
//
// Keys: the order-preserving image of the fp64 pattern of d (sign flipped
// for d >= 0, all bits flipped for d < 0), with its low 20 bits replaced by
// the neuron index. Comparing keys compares d (to 44 bits) and then the
// index, which gives the problem statement's lowest-index tie-break at every
// level of the reduction.

#pragma once

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

// The second word of a plan entry: the TA-bit mask of the tile's samples that hold
// the entry's feature. For tiles of up to 16 samples it also carries the slot of the
// lowest set bit (bits 24-28) and, in bit 31, whether more than one bit is set, so the
// sweep can send an entry held by one sample (most of them) straight to that
// sample's accumulators.
constexpr int kPlanSlotShift = 24;
constexpr unsigned kPlanMulti = 1u << 31;

template <int TA>
__device__ __forceinline__ unsigned plan_word(unsigned mask)
{
    if constexpr (TA <= 16)
        return mask | ((unsigned)__builtin_ctz(mask | (1u << 30)) << kPlanSlotShift) |
               ((mask & (mask - 1)) ? kPlanMulti : 0u);
    else
        return mask;
}

// The sample mask of a plan word.
template <int TA>
__device__ __forceinline__ unsigned plan_mask(unsigned y)
{
    if constexpr (TA < 32)
        return y & ((1u << TA) - 1u);
    else
        return y;
}

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

// First id offset of the batch, row_ptr[0] (col_idx is the base its offsets index). A
// negative one would name ids before col_idx: such a batch is read as empty (nnz = 0;
// its row pointers are then flagged as out of range wherever they are checked).
__device__ __forceinline__ int64_t csr_base(const int32_t *row_ptr, int64_t &nnz)
{
    const int64_t b = row_ptr[0];
    if (b < 0) {
        nnz = 0;
        return 0;
    }
    return b;
}

}  // namespace
}  // namespace som
