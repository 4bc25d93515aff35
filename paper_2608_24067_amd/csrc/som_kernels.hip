// som_kernels.hip -- gfx950 kernels of the sparse-binary BMU search other than the
// sweep (som_sweep.hip): the fp64 norms, the regrouping of the batch and the tile plan
// (Algorithm 2, step 5), and the finalize that reduces the sweep's per-strip keys.
//
// The plan (SpMM-tile kernel section) groups samples into tiles of TA consecutive
// rows and lists, per tile, the distinct feature ids of its rows in ascending order,
// each with a TA-bit mask of the rows holding it; the sweep (som_sweep.hip) streams
// those codebook rows once per tile and strip. Unless the caller keeps the sample
// order, the batch is first regrouped by each sample's least frequent feature (the
// post-submission section's lever of clustering samples so tiles share features).
// The finalize takes, per sample, the smallest of the sweep's per-strip keys and
// forms the winner's full squared distance from the dot product the sweep kept.

#include "som_device.h"

namespace som {
namespace {

// ----------------------------------------------------------------- norms

// n_i = sum_v W[v*M+i]^2: one thread per neuron, v ascending, fp64. The square of
// an fp32 (or fp16) value is exact in fp64, so fma(w, w, acc) equals acc + w*w.
// One wave per workgroup, so a small map (M = 4096: 64 waves) still spreads over
// 64 compute units, and NL rows in flight per wave: the sums are sequential, the
// loads are not. A map of fewer than kNormWavesFew waves is bound by each lane's
// chain of batches, so it takes 128 rows per batch (64x64 map: 0.64 -> 0.45 ms);
// larger maps keep 32 (128 costs 10% at 256x256, where 32 already reads at 7 TB/s).
constexpr int kNormWavesFew = 512;

template <typename E, int NL>
__global__ __launch_bounds__(64) void k_norms(const E *__restrict__ W, int64_t V, int64_t M,
                                              double *__restrict__ norms)
{
    constexpr int kNormLoads = NL;
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

// Row pointers checked before any kernel walks a row: non-decreasing and inside
// [row_ptr[0], row_ptr[0] + nnz], with row_ptr[0] >= 0. A batch that fails is flagged
// (SOM_FLAG_ROW_PTR) and every later kernel of the plan reads it as empty (rows_nnz),
// so row pointers that decrease cannot make rows overlap and multiply the work.
__global__ __launch_bounds__(256) void k_check_rows(const int32_t *__restrict__ row_ptr, int64_t N, int64_t nnz,
                                                    uint32_t *__restrict__ flags)
{
    const int64_t base = row_ptr[0];
    bool bad = base < 0;
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        const int64_t a = (int64_t)row_ptr[s] - base, b = (int64_t)row_ptr[s + 1] - base;
        if (b < a || a < 0 || b > nnz) bad = true;
    }
    if (__ballot(bad) != 0 && (threadIdx.x & 63) == 0) atomicOr(flags, SOM_FLAG_ROW_PTR);
}

// The ids a plan kernel may read: nnz, or none once the row pointers are flagged.
__device__ __forceinline__ int64_t rows_nnz(const uint32_t *flags, int64_t nnz)
{
    return (flags[0] & SOM_FLAG_ROW_PTR) ? 0 : nnz;
}

// ----------------------------------------------------------------- order

// Sample order. The post-submission section's tuning groups samples so that a
// tile's rows share features. Here the samples of a batch are bucketed by their
// least frequent feature in that batch: rows that share a rare feature land in
// the same or neighbouring tiles, which run close together in time, so a rare
// codebook row is re-read while still in L2. A sample's result does not depend on where it
// sits (its sum order is fixed by its own features), so the permutation never
// shows in the output. The permuted batch is written to the workspace as row offsets
// of its own and, per position, where that row's ids start in the caller's batch
// (both in pos, interleaved), from which the plan reads them; k_unpermute moves the results back
// to their samples.

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
    const int64_t base = csr_base(row_ptr, nnz);
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
// half, ids in the low half of one 64-bit word. The word the atomic returns is the
// sample's rank in its bucket (samples and ids before it), kept in rank[s]: once the
// buckets' starts are known it gives the sample's place without a second atomic.
__global__ __launch_bounds__(256) void k_rarest(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                                                int64_t N, int64_t nnz, int32_t V, const uint32_t *__restrict__ freq,
                                                int32_t *__restrict__ skey, u64 *__restrict__ bucket,
                                                u64 *__restrict__ rank,
                                                uint32_t *__restrict__ flags)
{
    // the four lanes of a quad share a row (lane q of the quad takes ids q, q + 4, ...)
    nnz = rows_nnz(flags, nnz);
    const int64_t base = csr_base(row_ptr, nnz);
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
            rank[s] = atomicAdd(&bucket[key], (1ull << 32) | (u64)(re - rb));
        }
    }
    if (bad) atomicOr(flags, bad);
}

// One workgroup: exclusive scan of the nb packed bucket counts into packed starting
// offsets (sample offset << 32 | id offset). *prp_end = total ids (capped at nnz).
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

// Sample s goes to its bucket's start plus its rank in the bucket (both packed as
// samples << 32 | ids; the id halves never carry): it sits at position inv[s] of the
// permuted batch, its ids at plan offsets pos[2 inv[s]] ..., and pos[2 inv[s] + 1] is where
// its row starts in the caller's col_idx (past row_ptr[0]). The rows themselves are
// not copied: the plan reads each position's ids from there. Positions past N and
// offsets past nnz (only reachable with invalid row pointers or a workspace the
// regrouping did not write) are dropped or clamped.
__global__ __launch_bounds__(256) void k_place(const int32_t *__restrict__ row_ptr, int64_t N, int64_t nnz,
                                               const int32_t *__restrict__ skey, const u64 *__restrict__ bucket,
                                               const u64 *__restrict__ rank, int64_t nb, int32_t *__restrict__ inv,
                                               int32_t *__restrict__ pos, const uint32_t *__restrict__ flags)
{
    nnz = rows_nnz(flags, nnz);
    const int64_t base = csr_base(row_ptr, nnz);
    for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < N; s += (int64_t)gridDim.x * 256) {
        const u64 at = bucket[clamp64(skey[s], 0, nb - 1)] + rank[s];
        const int64_t ps = (int64_t)(at >> 32), pi = (int64_t)(at & 0xFFFFFFFFull);
        inv[s] = ps < N ? (int32_t)ps : -1;
        if (ps >= N) continue;
        // one 8-byte word per sample: a scattered write costs a whole memory burst either way
        reinterpret_cast<int2 *>(pos)[ps] =
            make_int2((int32_t)(pi < nnz ? pi : nnz), (int32_t)clamp64((int64_t)row_ptr[s] - base, 0, nnz));
    }
}

// ------------------------------------------------------------------ plan

constexpr int kPlanWaves = 4;
// ids staged in LDS per wave: 16 KiB a workgroup (2048 would halve the workgroups a CU
// holds, 5% slower on the 64x64 workload)
constexpr int kPlanStage = 1024;

// A wave plans 64/TA consecutive tiles at once (TA = 2 ... 32): lane l works on row s = l % TA of
// tile l / TA. Each step takes, per tile, the smallest current id over its TA
// lanes (the next element of the union, ascending), the ballot of the lanes
// holding it (its sample mask), and advances those lanes: a TA-way merge of
// sorted lists per lane group. Offsets are clamped to [row_ptr[0], row_ptr[0]+nnz)
// and to each tile's own range, ids outside [0, V) are skipped, and a tile never
// writes more entries than its own CSR span, so no input can drive an access out
// of bounds.
//
// Offsets are read os words apart: off[p * os]. Regrouped batch (psrc non-null, os = 2):
// off (the regrouped row offsets) places every tile's entries and gives each position's
// row length; the row's ids start at psrc[p * os] in the caller's col_idx (past
// src_ptr[0]), clamped to the batch. Otherwise off is the caller's row_ptr (os = 1) and
// positions are samples.
//
// Real-valued rows (REAL, values given): every union entry also gets the TA values of
// its samples (vals[entry*TA + s], written for the samples whose mask bit is set;
// the other slots are never read), and every row the fp64 sum of its squared
// values in its own order (xsq, by batch position), which is ||x||^2.
template <int TA, bool REAL>
__global__ __launch_bounds__(256) void k_plan(const int32_t *__restrict__ off, int os,
                                              const int32_t *__restrict__ src_ptr, const int32_t *__restrict__ psrc,
                                              const int32_t *__restrict__ col_idx,
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
    nnz = rows_nnz(flags, nnz);
    const int64_t base = csr_base(off, nnz);
    const int64_t sbase = psrc ? csr_base(src_ptr, nnz) : base;
    uint32_t bad = 0;

    for (int64_t tb = (int64_t)blockIdx.x * kPlanWaves * G; tb < n_tiles; tb += (int64_t)gridDim.x * kPlanWaves * G) {
        const int64_t tw = tb + (int64_t)wv * G;  // first tile of this wave
        const int64_t t = tw + grp;               // this lane's tile
        const bool live = t < n_tiles;
        // the wave's CSR span, for staging
        int64_t wlo = 0, whi = 0;
        if (tw < n_tiles) {
            const int64_t te = tw + G < n_tiles ? tw + G : n_tiles;
            wlo = clamp64((int64_t)off[tw * TA * os] - base, 0, nnz);
            whi = clamp64((int64_t)off[(te * TA < N ? te * TA : N) * os] - base, wlo, nnz);
        }
        int64_t lo = 0, hi = 0, b = 0, e = 0;
        int64_t src = 0;  // where the lane's ids start in col_idx (past its base)
        if (live) {
            const int64_t s0 = t * TA;
            const int64_t s1 = s0 + TA < N ? s0 + TA : N;
            lo = clamp64((int64_t)off[s0 * os] - base, wlo, whi);
            hi = clamp64((int64_t)off[s1 * os] - base, lo, whi);
            if (s0 + sl < N) {
                const int64_t rb = (int64_t)off[(s0 + sl) * os] - base;
                const int64_t re = (int64_t)off[(s0 + sl + 1) * os] - base;
                if (re < rb || rb < lo || re > hi) bad |= SOM_FLAG_ROW_PTR;
                b = clamp64(rb, lo, hi);
                e = clamp64(re, b, hi);
                src = b;
                if (psrc) {
                    // the caller's row at this position (its flags were set by the regrouping),
                    // never reaching past the batch
                    src = clamp64(psrc[(s0 + sl) * os], 0, nnz);
                    if (nnz - src < e - b) e = b + (nnz - src);
                }
            }
        }
        const bool staged = (whi - wlo) <= kPlanStage;  // wave-uniform
        if (staged) {
            if (psrc) {
                for (int64_t q = 0; q < e - b; ++q) stage[wv][b - wlo + q] = col_idx[sbase + src + q];
            } else {
                for (int64_t q = lane; q < whi - wlo; q += 64) stage[wv][q] = col_idx[base + wlo + q];
            }
        }
        __syncthreads();

        // positions in 32 bits: every offset lies in [0, nnz] and nnz < 2^31
        const int64_t shift = sbase + src - b;  // the lane's id q (b <= q < e) is col_idx[shift + q]
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
                    return col_idx[shift + q];
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
                    curv = values[shift + p];
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
                        if (sl == 0) plan[plo + k] = make_uint2((unsigned)m, plan_word<TA>(mask));
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
                                                  const int32_t *__restrict__ row_ptr, int rs, int64_t N, int64_t nnz,
                                                  const double *__restrict__ xsq,
                                                  const u64 *__restrict__ keys,
                                                  const float *__restrict__ dots, int64_t n_strips,
                                                  FinalOut out)
{
    const int64_t base = csr_base(row_ptr, nnz);
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
        const int64_t rb = clamp64((int64_t)row_ptr[k * rs] - base, 0, nnz);
        const int64_t re = clamp64((int64_t)row_ptr[(k + 1) * rs] - base, rb, nnz);
        out.put(k, (int32_t)b, fma(-2.0, (double)dots[gb * N + k], norms[b]) + (xsq ? xsq[k] : (double)(re - rb)));
    }
}

// Two best units: the two smallest of the 2 * n_strips keys of each sample (each
// strip's two smallest), with their dot products from the sweep. Without a second
// unit (M == 1) bmu2 = -1 and dist2 = +inf.
__global__ __launch_bounds__(256) void k_finalize2(const double *__restrict__ norms, int64_t M,
                                                   const int32_t *__restrict__ row_ptr, int rs, int64_t N, int64_t nnz,
                                                   const double *__restrict__ xsq,
                                                   const u64 *__restrict__ keys,
                                                   const float *__restrict__ dots, const u64 *__restrict__ keys2,
                                                   const float *__restrict__ dots2, int64_t n_strips,
                                                   FinalOut out, FinalOut out2)
{
    const int64_t base = csr_base(row_ptr, nnz);
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
        const int64_t rb = clamp64((int64_t)row_ptr[k * rs] - base, 0, nnz);
        const int64_t re = clamp64((int64_t)row_ptr[(k + 1) * rs] - base, rb, nnz);
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
    if (blocks < kNormWavesFew)
        hipLaunchKernelGGL((k_norms<float, 128>), dim3((unsigned)blocks), dim3(64), 0, st, W, V, M, norms);
    else
        hipLaunchKernelGGL((k_norms<float, 32>), dim3((unsigned)blocks), dim3(64), 0, st, W, V, M, norms);
    return hipGetLastError();
}

hipError_t launch_norms_f16(const uint16_t *W, int64_t V, int64_t M, double *norms, hipStream_t st)
{
    const int64_t blocks = (M + 63) / 64;
    const _Float16 *w = reinterpret_cast<const _Float16 *>(W);
    if (blocks < kNormWavesFew)
        hipLaunchKernelGGL((k_norms<_Float16, 128>), dim3((unsigned)blocks), dim3(64), 0, st, w, V, M, norms);
    else
        hipLaunchKernelGGL((k_norms<_Float16, 32>), dim3((unsigned)blocks), dim3(64), 0, st, w, V, M, norms);
    return hipGetLastError();
}

hipError_t launch_clear_flags(uint32_t *flags, hipStream_t st)
{
    hipLaunchKernelGGL(k_clear_flags, dim3(1), dim3(64), 0, st, flags);
    return hipGetLastError();
}

hipError_t launch_check_rows(const int32_t *row_ptr, int64_t N, int64_t nnz, uint32_t *flags, hipStream_t st)
{
    int64_t blocks = (N + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_check_rows, dim3((unsigned)blocks), dim3(256), 0, st, row_ptr, N, nnz, flags);
    return hipGetLastError();
}

hipError_t launch_plan(int ta, const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N,
                       int64_t nnz, int64_t V, const OrderBuffers *ob, uint2 *plan, int2 *tiles, float *vals,
                       double *xsq, uint32_t *flags, hipStream_t st)
{
    const int64_t nt = n_tiles(N, ta);
    const int64_t per_block = (int64_t)kPlanWaves * (64 / ta);
    int64_t blocks = (nt + per_block - 1) / per_block;
    if (blocks > (1 << 22)) blocks = 1 << 22;
    const dim3 grid((unsigned)blocks), block(256);
    const int32_t v = (int32_t)V;
    // a regrouped batch's offsets and sources are interleaved in ob->pos
    const int32_t *off = ob ? ob->pos : row_ptr;
    const int32_t *psrc = ob ? ob->pos + 1 : nullptr;
    const int os = ob ? 2 : 1;
    if (values) {  // real-valued rows: tiles of 8 only
        if (ta != 8) return hipErrorInvalidValue;
        hipLaunchKernelGGL((k_plan<8, true>), grid, block, 0, st, off, os, row_ptr, psrc, col_idx, N, nnz, v, nt,
                           plan, tiles, flags, values, vals, xsq);
        return hipGetLastError();
    }
    switch (ta) {
    case 8:
        hipLaunchKernelGGL((k_plan<8, false>), grid, block, 0, st, off, os, row_ptr, psrc, col_idx, N, nnz, v, nt,
                           plan, tiles, flags, nullptr, nullptr, nullptr);
        break;
    case 16:
        hipLaunchKernelGGL((k_plan<16, false>), grid, block, 0, st, off, os, row_ptr, psrc, col_idx, N, nnz, v, nt,
                           plan, tiles, flags, nullptr, nullptr, nullptr);
        break;
    case 32:
        hipLaunchKernelGGL((k_plan<32, false>), grid, block, 0, st, off, os, row_ptr, psrc, col_idx, N, nnz, v, nt,
                           plan, tiles, flags, nullptr, nullptr, nullptr);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_finalize(int ta, const double *norms, int64_t M, const int32_t *row_ptr, int64_t N, int64_t nnz,
                           const OrderBuffers *ob, const double *xsq, const SweepOut &o, int32_t *bmu, double *dist,
                           int32_t *bmu2, double *dist2, hipStream_t st)
{
    int64_t blocks = (N + 255) / 256;
    if (blocks > (1 << 22)) blocks = 1 << 22;
    // a regrouped batch is finalized by position into the workspace first, with its row
    // lengths from the interleaved offsets of its positions
    const FinalOut o1{bmu, dist, ob ? ob->res : nullptr}, o2{bmu2, dist2, ob ? ob->res2 : nullptr};
    const int32_t *rp = ob ? ob->pos : row_ptr;
    const int rs = ob ? 2 : 1;
    if (bmu2)
        hipLaunchKernelGGL(k_finalize2, dim3((unsigned)blocks), dim3(256), 0, st, norms, M, rp, rs, N, nnz, xsq,
                           o.keys, o.dots, o.keys2, o.dots2, n_strips(M, ta), o1, o2);
    else
        hipLaunchKernelGGL(k_finalize, dim3((unsigned)blocks), dim3(256), 0, st, norms, M, rp, rs, N, nnz, xsq,
                           o.keys, o.dots, n_strips(M, ta), o1);
    if (ob)
        hipLaunchKernelGGL(k_unpermute, dim3((unsigned)blocks), dim3(256), 0, st, ob->inv, N, ob->res,
                           bmu2 ? ob->res2 : nullptr, bmu, dist, bmu2, dist2);
    return hipGetLastError();
}

hipError_t launch_order(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz, int64_t V,
                        const OrderBuffers &ob, uint32_t *flags, hipStream_t st)
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
                       ob.skey, ob.bucket, ob.rank, flags);
    hipLaunchKernelGGL(k_bucket_scan, dim3(1), dim3(1024), 0, st, ob.bucket, nb, nnz, ob.pos + 2 * N);
    int64_t pb = (N + 255) / 256;
    if (pb > (1 << 22)) pb = 1 << 22;
    hipLaunchKernelGGL(k_place, dim3((unsigned)pb), dim3(256), 0, st, row_ptr, N, nnz, ob.skey, ob.bucket, ob.rank, nb,
                       ob.inv, ob.pos, flags);
    return hipGetLastError();
}

}  // namespace som
