// som_update.hip -- gfx950 kernels of the batch-SOM update (Algorithm 2, steps 8-9;
// factorised box-blur update section), for binary rows.
//
// After a search has given every sample its best unit, the update
//   1. scatters the batch onto the E x E lattice: den[i] = samples at unit i and,
//      feature by feature, num[v][i] = samples at unit i holding feature v (integer
//      counts: exact and independent of the order they are taken in). Units that
//      hold many samples (on an untrained codebook a handful of units can take the
//      whole batch) are counted in LDS: their samples are sorted by unit and each
//      workgroup histograms a run of one unit's samples, then adds the non-zero
//      bins to global memory; the other units take one global atomic per feature.
//      The counts are unit-major (cnt[i][v]), and so are the blurred fields: in
//      every pass neighbouring lanes take neighbouring features;
//   2. converts both fields to fp32 and blurs them: three box passes along every
//      lattice row, then three along every lattice column, each a running window
//      sum over the clamped window (the first window summed in ascending order,
//      then per step the element entering added and the one leaving subtracted),
//      unnormalised -- the constant cancels in the quotient;
//   3. replaces every prototype by num / den (fp32 division), clamped to [0, 1] (a
//      mean of 0/1 inputs), leaving a unit unchanged where no sample lies in its
//      neighbourhood; an fp16 codebook receives the quotient rounded once to
//      binary16 at this final write. In exact arithmetic the blurred den is zero
//      exactly where no unit within 3r cells along both axes holds a sample, but
//      fp32 running sums past 2^24 can leave a residual there, so that support is
//      counted separately in whole numbers (k_support) and decides the rule.
// A lane owns one lattice line (row or column) of one field and runs its three
// passes in one sweep of the line, each pass exactly in the order above, so the
// result is the same bits on every run; the blurred field replaces the counts.
// The quotient is fused with the one transpose, from the unit-major fields to the
// feature-major codebook. Features are processed in
// chunks, so the workspace holds three fields of chunk * M values rather than V * M.

#include <climits>

#include "../../include/som.h"
#include "som_internal.h"

namespace som {
namespace {

typedef unsigned long long u64;

// A unit with at least kHeavy samples is counted through LDS; kRunSamples sorted
// samples per workgroup there, and kLdsBins feature bins (64 KB) per LDS pass.
constexpr int32_t kHeavy = 1024;
constexpr int64_t kRunSamples = 16384;
constexpr int kLdsBins = 16384;

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// Clamped id range of sample s (relative to row_ptr[0]).
__device__ __forceinline__ void sample_ids(const int32_t *row_ptr, int64_t base, int64_t nnz, int64_t s, int64_t &rb,
                                           int64_t &re)
{
    rb = (int64_t)row_ptr[s] - base;
    re = (int64_t)row_ptr[s + 1] - base;
    rb = rb < 0 ? 0 : (rb > nnz ? nnz : rb);
    re = re < rb ? rb : (re > nnz ? nnz : re);
}

// Each wave takes a contiguous range of samples, 64 at a time; kScanBlocks blocks.
constexpr int64_t kScanBlocks = 2048;

__device__ __forceinline__ void wave_range(int64_t N, int64_t &w0, int64_t &w1)
{
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    const int64_t w = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    const int64_t per = ((N + waves - 1) / waves + 63) / 64 * 64;
    w0 = w * per < N ? w * per : N;
    w1 = w0 + per < N ? w0 + per : N;
}

// Samples per unit. The lanes of a wave that share a unit add their count with one
// atomic, and a wave carries a unit's count over as long as consecutive samples keep
// it, so a unit that takes most of the batch does not serialise the grid on one
// address.
__global__ __launch_bounds__(256) void k_count_units(const int32_t *__restrict__ bmu, int64_t N, int64_t M,
                                                     int32_t *__restrict__ cnt)
{
    const int lane = lane_id();
    int64_t w0, w1;
    wave_range(N, w0, w1);
    int32_t pu = -1, pn = 0;  // the unit whose count is carried, and the count (wave-uniform)
    for (int64_t s0 = w0; s0 < w1; s0 += 64) {
        const int64_t s = s0 + lane;
        int32_t u = -1;
        if (s < w1) {
            u = bmu[s];
            if (u < 0 || u >= M) u = -1;
        }
        u64 todo = __ballot(u >= 0);
        while (todo) {
            const int leader = __builtin_ctzll(todo);
            const int32_t lu = __builtin_amdgcn_readlane(u, leader);
            const u64 same = __ballot(u == lu) & todo;
            if (lu == pu) {
                pn += (int32_t)__popcll(same);
            } else {
                if (pu >= 0 && lane == 0) atomicAdd(cnt + pu, pn);
                pu = lu;
                pn = (int32_t)__popcll(same);
            }
            todo &= ~same;
        }
    }
    if (pu >= 0 && lane == 0) atomicAdd(cnt + pu, pn);
}

// Samples per unit for maps of at most kLdsUnits units: a histogram in LDS per
// workgroup (1024 threads), then one global atomic per non-zero bin.
constexpr int kLdsUnits = 16384;

__global__ __launch_bounds__(1024) void k_count_units_lds(const int32_t *__restrict__ bmu, int64_t N, int64_t M,
                                                          int32_t *__restrict__ cnt)
{
    __shared__ uint32_t h[kLdsUnits];
    for (int64_t i = threadIdx.x; i < M; i += 1024) h[i] = 0u;
    __syncthreads();
    for (int64_t s = (int64_t)blockIdx.x * 1024 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 1024) {
        const int32_t u = bmu[s];
        if (u >= 0 && u < M) atomicAdd(&h[u], 1u);
    }
    __syncthreads();
    for (int64_t i = threadIdx.x; i < M; i += 1024)
        if (h[i]) atomicAdd(cnt + i, (int32_t)h[i]);
}

// One workgroup: start[u] = number of samples of heavy units below u (heavy: at least
// kHeavy samples), start[M] = all samples of heavy units, start[M + 1] = number of
// heavy units; cursor = start; slot[u] = the heavy unit's rank among heavy units (-1
// for the others) and hunit[slot] = u.
__global__ __launch_bounds__(1024) void k_heavy_scan(const int32_t *__restrict__ cnt, int64_t M,
                                                     int32_t *__restrict__ start, int32_t *__restrict__ cursor,
                                                     int32_t *__restrict__ slot, int32_t *__restrict__ hunit)
{
    __shared__ int64_t ss[1024], sk[1024];
    const int t = threadIdx.x;
    const int64_t per = (M + 1023) / 1024;
    const int64_t b0 = t * per < M ? t * per : M;
    const int64_t b1 = b0 + per < M ? b0 + per : M;
    int64_t n = 0, k = 0;
    for (int64_t u = b0; u < b1; ++u)
        if (cnt[u] >= kHeavy) {
            n += cnt[u];
            ++k;
        }
    ss[t] = n;
    sk[t] = k;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {  // inclusive Hillis-Steele scans
        const int64_t a = t >= d ? ss[t - d] : 0, c = t >= d ? sk[t - d] : 0;
        __syncthreads();
        ss[t] += a;
        sk[t] += c;
        __syncthreads();
    }
    int64_t o = ss[t] - n, q = sk[t] - k;
    for (int64_t u = b0; u < b1; ++u) {
        start[u] = (int32_t)o;
        cursor[u] = (int32_t)o;
        if (cnt[u] >= kHeavy) {
            o += cnt[u];
            slot[u] = (int32_t)q;
            hunit[q] = (int32_t)u;
            ++q;
        } else {
            slot[u] = -1;
        }
    }
    if (t == 1023) {
        start[M] = (int32_t)ss[1023];
        start[M + 1] = (int32_t)sk[1023];
    }
}

// order[start[u] ...] = the samples of every heavy unit u, grouped by unit (in any
// order within a unit: the counts do not depend on it). A workgroup (1024 threads)
// takes a contiguous range of samples. With at most kLdsUnits heavy units it counts
// them per heavy unit in LDS, reserves each unit's positions with one global atomic,
// and hands them out from LDS in a second pass over the range. Otherwise each wave
// reserves, per 64 samples, one run of positions per distinct unit.
__global__ __launch_bounds__(1024) void k_heavy_scatter(const int32_t *__restrict__ bmu, int64_t N, int64_t M,
                                                        const int32_t *__restrict__ start,
                                                        const int32_t *__restrict__ slot,
                                                        const int32_t *__restrict__ hunit, int32_t *__restrict__ cursor,
                                                        int32_t *__restrict__ order)
{
    __shared__ int32_t h[kLdsUnits];
    const int64_t per = (N + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = (int64_t)blockIdx.x * per < N ? (int64_t)blockIdx.x * per : N;
    const int64_t b1 = b0 + per < N ? b0 + per : N;
    const int32_t heavy = start[M + 1];
    auto slot_of = [&](int64_t s) {
        const int32_t u = bmu[s];
        return u >= 0 && u < M ? slot[u] : -1;
    };
    if (heavy <= kLdsUnits) {  // uniform
        for (int i = threadIdx.x; i < heavy; i += 1024) h[i] = 0;
        __syncthreads();
        for (int64_t s = b0 + threadIdx.x; s < b1; s += 1024) {
            const int32_t k = slot_of(s);
            if (k >= 0 && k < heavy) atomicAdd(&h[k], 1);
        }
        __syncthreads();
        for (int i = threadIdx.x; i < heavy; i += 1024)
            if (h[i]) h[i] = atomicAdd(cursor + hunit[i], h[i]);
        __syncthreads();
        for (int64_t s = b0 + threadIdx.x; s < b1; s += 1024) {
            const int32_t k = slot_of(s);
            if (k >= 0 && k < heavy) order[atomicAdd(&h[k], 1)] = (int32_t)s;
        }
        return;
    }
    const int lane = lane_id();
    const u64 below = (1ull << lane) - 1ull;
    const int64_t wb = b0 + (int64_t)(threadIdx.x >> 6) * 64;
    for (int64_t s0 = wb; s0 < b1; s0 += 1024) {
        const int64_t s = s0 + lane;
        int32_t u = -1;
        if (s < b1) {
            u = bmu[s];
            if (u < 0 || u >= M || slot[u] < 0) u = -1;
        }
        u64 todo = __ballot(u >= 0);
        while (todo) {
            const int leader = __builtin_ctzll(todo);
            const int32_t lu = __builtin_amdgcn_readlane(u, leader);
            const u64 same = __ballot(u == lu) & todo;
            int32_t at = 0;
            if (lane == leader) at = atomicAdd(cursor + lu, (int32_t)__popcll(same));
            at = __builtin_amdgcn_readlane(at, leader);
            if ((same >> lane) & 1ull) order[at + __popcll(same & below)] = (int32_t)s;
            todo &= ~same;
        }
    }
}

// cnt[u][v - v0] += 1 (unit-major, f = v1 - v0 per unit) for every id v in [v0, v1)
// of every sample whose unit is not heavy.
__global__ __launch_bounds__(256) void k_count_light(const int32_t *__restrict__ row_ptr,
                                                     const int32_t *__restrict__ col_idx, int64_t N, int64_t nnz,
                                                     const int32_t *__restrict__ bmu, int64_t M,
                                                     const int32_t *__restrict__ units, int32_t v0, int32_t v1,
                                                     int32_t *__restrict__ cnt, const uint32_t *__restrict__ flags)
{
    if (flags[0] & SOM_FLAG_ROW_PTR) return;  // invalid row pointers: no row is read
    const int64_t base = row_ptr[0];           // >= 0 once the row pointers passed the check
    const int64_t f = (int64_t)v1 - v0;
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        const int32_t u = bmu[s];
        if (u < 0 || u >= M || units[u] >= kHeavy) continue;
        int64_t rb, re;
        sample_ids(row_ptr, base, nnz, s, rb, re);
        for (int64_t p = rb; p < re; ++p) {
            const int32_t v = col_idx[base + p];
            if (v >= v0 && v < v1) atomicAdd(cnt + (int64_t)u * f + (v - v0), 1);
        }
    }
}

// Heavy units: workgroup b takes the sorted positions [b * kRunSamples, ...) of
// order; each run of one unit's samples in that range is histogrammed in LDS, in
// passes of kLdsBins features, and the non-zero bins are added to cnt[u][.].
__global__ __launch_bounds__(256) void k_count_heavy(const int32_t *__restrict__ row_ptr,
                                                     const int32_t *__restrict__ col_idx, int64_t nnz,
                                                     const int32_t *__restrict__ bmu, int64_t M,
                                                     const int32_t *__restrict__ units,
                                                     const int32_t *__restrict__ start,
                                                     const int32_t *__restrict__ order, int32_t v0, int32_t v1,
                                                     int32_t *__restrict__ cnt, const uint32_t *__restrict__ flags)
{
    __shared__ uint32_t hist[kLdsBins];
    if (flags[0] & SOM_FLAG_ROW_PTR) return;  // uniform: invalid row pointers, no row is read
    const int64_t base = row_ptr[0];           // >= 0 once the row pointers passed the check
    const int64_t f = (int64_t)v1 - v0;
    const int64_t total = start[M];
    const int64_t p0 = (int64_t)blockIdx.x * kRunSamples;
    if (p0 >= total) return;  // uniform
    const int64_t p1 = p0 + kRunSamples < total ? p0 + kRunSamples : total;
    for (int64_t p = p0; p < p1;) {  // uniform: every thread reads the same run bounds
        const int32_t u = bmu[order[p]];
        int64_t re = p + 1;
        if (u >= 0 && u < M) {
            const int64_t end = (int64_t)start[u] + units[u];
            re = end < p1 ? end : p1;
            if (re <= p) re = p + 1;
        }
        if (u >= 0 && u < M) {
            for (int64_t h0 = v0; h0 < v1; h0 += kLdsBins) {
                const int hb = (int)((int64_t)v1 - h0 < kLdsBins ? (int64_t)v1 - h0 : kLdsBins);
                for (int b = threadIdx.x; b < hb; b += 256) hist[b] = 0u;
                __syncthreads();
                for (int64_t q = p + threadIdx.x; q < re; q += 256) {
                    int64_t rb, rend;
                    sample_ids(row_ptr, base, nnz, order[q], rb, rend);
                    for (int64_t k = rb; k < rend; ++k) {
                        const int64_t v = col_idx[base + k];
                        if (v >= h0 && v < h0 + hb) atomicAdd(&hist[v - h0], 1u);
                    }
                }
                __syncthreads();
                for (int b = threadIdx.x; b < hb; b += 256) {
                    const uint32_t c = hist[b];
                    if (c) atomicAdd(cnt + (int64_t)u * f + (h0 - v0 + b), (int32_t)c);
                }
                __syncthreads();
            }
        }
        p = re;
    }
}

// Three running-sum box passes of half-width r along lines of n values, `stride`
// apart, in one sweep of each line. Pass k+1 takes every value of pass k as pass k
// produces it -- that is the value entering pass k+1's window -- and reads the value
// leaving its window back from where pass k stored it (x holds pass 1's output, y
// pass 2's). Each pass is still exactly the oracle's sequence of fp32 operations: its
// first window summed in ascending order, then per step the entering value added and
// the leaving one subtracted. Per element that is four reads and three writes, where
// three separate passes take six reads and three writes.
// in holds the first pass's input as 32-bit words: integer counts (INT) or float
// bits. out receives the third pass as float bits and may be in itself: out[i] is
// written once pass 1 has gone past i + 2m (m = min(r, n - 1)), after its last read
// of in[i] at i + r + 1. The words are read and written through one type, so no
// access to in and out can be reordered across another.
// Fields are unit-major: element (r, c) of feature v is at (r * E + c) * f + v. Line
// l is feature v = l % f of the line k = l / f and starts at k * outer + v;
// neighbouring lanes take neighbouring features, so every step is one coalesced
// access per lane group. Row passes (along c): outer = E * f, stride = f; column
// passes (along r): outer = f, stride = E * f. The lines of different lanes are
// disjoint.
template <bool INT>
__global__ __launch_bounds__(256) void k_blur3(const uint32_t *in, float *x, float *y, uint32_t *out, int64_t lines,
                                               int64_t f, int64_t outer, int64_t n, int64_t stride, int64_t r)
{
    for (int64_t l = (int64_t)blockIdx.x * 256 + threadIdx.x; l < lines; l += (int64_t)gridDim.x * 256) {
        const int64_t off = (l / f) * outer + l % f;
        const uint32_t *src = in + off;
        float *px = x + off, *py = y + off;
        uint32_t *dst = out + off;
        auto input = [&](int64_t k) {
            const uint32_t u = src[k * stride];
            return INT ? (float)(int32_t)u : __uint_as_float(u);
        };
        const int64_t m = r < n - 1 ? r : n - 1;  // the first window is [0, m]
        float s1 = 0.0f, s2 = 0.0f;
        int64_t next1 = 0, next2 = 0;  // the next output index of passes 2 and 3
        // pass 3 receives pass 2's output j
        auto feed2 = [&](int64_t j, float v) {
            py[j * stride] = v;
            s2 += v;
            if (j >= m) {  // output i = j - m: its first window is complete, or v entered at i + r
                const int64_t i = j - m;
                if (i - r - 1 >= 0) s2 -= py[(i - r - 1) * stride];
                dst[i * stride] = __float_as_uint(s2);
                next2 = i + 1;
            }
        };
        // pass 2 receives pass 1's output j
        auto feed1 = [&](int64_t j, float v) {
            px[j * stride] = v;
            s1 += v;
            if (j >= m) {
                const int64_t i = j - m;
                if (i - r - 1 >= 0) s1 -= px[(i - r - 1) * stride];
                feed2(i, s1);
                next1 = i + 1;
            }
        };
        // pass 1
        float s0 = 0.0f;
        for (int64_t k = 0; k <= m; ++k) s0 += input(k);
        feed1(0, s0);
        for (int64_t i = 1; i < n; ++i) {
            if (i + r < n) s0 += input(i + r);
            if (i - r - 1 >= 0) s0 -= input(i - r - 1);
            feed1(i, s0);
        }
        // passes 2 and 3 past the last entering value: only leaving values remain
        for (int64_t i = next1; i < n; ++i) {
            if (i - r - 1 >= 0) s1 -= px[(i - r - 1) * stride];
            feed2(i, s1);
        }
        for (int64_t i = next2; i < n; ++i) {
            if (i - r - 1 >= 0) s2 -= py[(i - r - 1) * stride];
            dst[i * stride] = __float_as_uint(s2);
        }
    }
}

// Occupied units counted over windows of half-width R along lattice lines, one lane per
// line: rows (in = the den counts, counted where > 0; out[r][c] = occupied units in row r
// within R of column c), then columns (in = the row counts, summed). Whole numbers, exact.
__global__ __launch_bounds__(256) void k_support(const int32_t *__restrict__ in, int32_t *__restrict__ out,
                                                 int64_t E, int64_t R, int rows)
{
    const int64_t l = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (l >= E) return;
    const int64_t first = rows ? l * E : l, step = rows ? 1 : E;
    auto val = [&](int64_t j) { return rows ? (in[first + j * step] > 0 ? 1 : 0) : in[first + j * step]; };
    int32_t s = 0;
    for (int64_t j = 0; j <= R && j < E; ++j) s += val(j);
    out[first] = s;
    for (int64_t i = 1; i < E; ++i) {
        if (i + R < E) s += val(i + R);
        if (i - R - 1 >= 0) s -= val(i - R - 1);
        out[first + i * step] = s;
    }
}

// W[v0 + v][i] = num[i][v] / den[i], clamped to [0, 1], where unit i has a sample in its
// neighbourhood (sup[i] > 0) and den[i] > 0 (fp32; rounded once to binary16 for an fp16
// codebook), unchanged elsewhere: the quotient fused with the transpose from unit-major
// to feature-major, in 64 (units) x 64 (features) tiles through LDS.
template <typename E>
__global__ __launch_bounds__(256) void k_quotient_t(E *__restrict__ W, const float *__restrict__ num,
                                                    const float *__restrict__ den, const int32_t *__restrict__ sup,
                                                    int64_t f, int64_t M, int64_t v0, const uint32_t *__restrict__ flags)
{
    __shared__ float tile[64][65];
    if (flags[0] & SOM_FLAG_ROW_PTR) return;  // uniform: invalid row pointers leave the codebook as it is
    const int64_t it = (M + 63) / 64, vt = (f + 63) / 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4 threads
    for (int64_t t = blockIdx.x; t < it * vt; t += gridDim.x) {
        const int64_t i0 = (t / vt) * 64, w0 = (t % vt) * 64;
        for (int y = ty; y < 64; y += 4)
            if (i0 + y < M && w0 + tx < f) tile[y][tx] = num[(i0 + y) * f + w0 + tx];
        __syncthreads();
        if (i0 + tx < M) {
            const float d = den[i0 + tx];
            if (sup[i0 + tx] > 0 && d > 0.0f)
                for (int y = ty; y < 64; y += 4)
                    if (w0 + y < f) W[(v0 + w0 + y) * M + i0 + tx] = (E)fminf(fmaxf(tile[tx][y] / d, 0.0f), 1.0f);
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void k_zero_i32(int32_t *__restrict__ p, int64_t n)
{
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256) p[k] = 0;
}

unsigned grid_for(int64_t n)
{
    int64_t b = (n + 255) / 256;
    if (b < 1) b = 1;
    if (b > (1 << 20)) b = 1 << 20;
    return (unsigned)b;
}

// The blur of f unit-major lattices (E x E) of counts: three row passes, then three
// column passes, with a and b as the passes' scratch. Result in out (fp32), which
// may be the counts themselves.
void blur(const int32_t *cnt, float *a, float *b, float *out, int64_t f, int64_t E, int64_t r, hipStream_t st)
{
    const unsigned g = grid_for(f * E);
    const uint32_t *in = reinterpret_cast<const uint32_t *>(cnt);
    uint32_t *o = reinterpret_cast<uint32_t *>(out);
    hipLaunchKernelGGL(k_blur3<true>, dim3(g), dim3(256), 0, st, in, a, b, o, f * E, f, E * f, E, f, r);
    hipLaunchKernelGGL(k_blur3<false>, dim3(g), dim3(256), 0, st, o, a, b, o, f * E, f, f, E, E * f, r);
}

}  // namespace

hipError_t launch_update(bool f16, void *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx,
                         int64_t N, int64_t nnz, const int32_t *bmu, int64_t radius, int64_t chunk,
                         const UpdateBuffers &ub, hipStream_t st)
{
    const int64_t M = E * E;
    // row pointers checked before any row is read: a batch that fails updates nothing
    hipError_t e = launch_clear_flags(ub.flags, st);
    if (e == hipSuccess) e = launch_check_rows(row_ptr, N, nnz, ub.flags, st);
    if (e != hipSuccess) return e;
    // den: counts, blur, kept in ub.den_blur; the samples of heavy units sorted by unit
    const unsigned sg = (unsigned)((N + 255) / 256 < kScanBlocks ? (N + 255) / 256 + 1 : kScanBlocks);
    const unsigned lg = (unsigned)((N + 1023) / 1024 < 512 ? (N + 1023) / 1024 + 1 : 512);
    hipLaunchKernelGGL(k_zero_i32, dim3(grid_for(M)), dim3(256), 0, st, ub.den_cnt, M);
    if (M <= kLdsUnits)
        hipLaunchKernelGGL(k_count_units_lds, dim3(lg), dim3(1024), 0, st, bmu, N, M, ub.den_cnt);
    else
        hipLaunchKernelGGL(k_count_units, dim3(sg), dim3(256), 0, st, bmu, N, M, ub.den_cnt);
    hipLaunchKernelGGL(k_heavy_scan, dim3(1), dim3(1024), 0, st, ub.den_cnt, M, ub.start, ub.cursor, ub.slot,
                       ub.hunit);
    hipLaunchKernelGGL(k_heavy_scatter, dim3(lg), dim3(1024), 0, st, bmu, N, M, ub.start, ub.slot, ub.hunit, ub.cursor,
                       ub.order);
    blur(ub.den_cnt, ub.den_a, ub.den_b, ub.den_blur, 1, E, radius, st);
    const unsigned lines = (unsigned)((E + 255) / 256);
    hipLaunchKernelGGL(k_support, dim3(lines), dim3(256), 0, st, ub.den_cnt, ub.sup_row, E, 3 * radius, 1);
    hipLaunchKernelGGL(k_support, dim3(lines), dim3(256), 0, st, ub.sup_row, ub.sup, E, 3 * radius, 0);
    const int64_t runs = (N + kRunSamples - 1) / kRunSamples;
    for (int64_t v0 = 0; v0 < V; v0 += chunk) {
        const int64_t f = V - v0 < chunk ? V - v0 : chunk;
        hipLaunchKernelGGL(k_zero_i32, dim3(grid_for(f * M)), dim3(256), 0, st, ub.cnt, f * M);
        hipLaunchKernelGGL(k_count_light, dim3(grid_for(N)), dim3(256), 0, st, row_ptr, col_idx, N, nnz, bmu, M,
                           ub.den_cnt, (int32_t)v0, (int32_t)(v0 + f), ub.cnt, ub.flags);
        if (runs > 0)
            hipLaunchKernelGGL(k_count_heavy, dim3((unsigned)runs), dim3(256), 0, st, row_ptr, col_idx, nnz, bmu, M,
                               ub.den_cnt, ub.start, ub.order, (int32_t)v0, (int32_t)(v0 + f), ub.cnt, ub.flags);
        float *num = reinterpret_cast<float *>(ub.cnt);  // the blur's result replaces the counts
        blur(ub.cnt, ub.a, ub.b, num, f, E, radius, st);
        const int64_t qt = ((M + 63) / 64) * ((f + 63) / 64);
        const unsigned qg = (unsigned)(qt < (1 << 20) ? qt : (1 << 20));
        if (f16)
            hipLaunchKernelGGL(k_quotient_t<_Float16>, dim3(qg), dim3(256), 0, st, static_cast<_Float16 *>(W), num,
                               ub.den_blur, ub.sup, f, M, v0, ub.flags);
        else
            hipLaunchKernelGGL(k_quotient_t<float>, dim3(qg), dim3(256), 0, st, static_cast<float *>(W), num,
                               ub.den_blur, ub.sup, f, M, v0, ub.flags);
    }
    return hipGetLastError();
}

}  // namespace som
