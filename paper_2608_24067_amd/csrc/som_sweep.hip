// som_sweep.hip -- the fused sweep of the sparse-binary BMU search (gfx950).
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

#include "som_device.h"
#include "som_tree16.h"
#include "som_tree8.h"

namespace som {
namespace {

// ----------------------------------------------------------------- sweep

// Tiles of 8 with eight neurons per lane keep four waves per SIMD (128 registers): the
// assembly dispatch of fp16 and real-valued rows would otherwise take up to 133 and
// lose a wave.
template <typename E, int TA, int NPL, bool VEC, bool REAL>
constexpr int sweep_min_waves()
{
    return (TA == 8 && NPL == 8 && VEC) ? 4 : 1;
}

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
__global__ __launch_bounds__(256, (sweep_min_waves<E, TA, NPL, VEC, REAL>())) void k_sweep(
    const E *__restrict__ W, const double *__restrict__ norms, int64_t M, int64_t N, int64_t V, int64_t nnz,
    const uint2 *__restrict__ plan, const int2 *__restrict__ tiles, int64_t n_tiles, u64 *__restrict__ keys,
    float *__restrict__ dots, u64 *__restrict__ keys2, float *__restrict__ dots2, const float *__restrict__ vals,
    int64_t group_tiles)
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
    // Tiles of 16 with four fp32 neurons per lane: the row dispatch is one assembly
    // block per row (som_tree16.h), and a row's address is one vector multiply-add
    // from the lane's own start of the strip (the row pitch is kept in a vector
    // register for that), which leaves the scalar unit to the dispatch.
    constexpr bool T16 = sizeof(E) == 4 && TA == 16 && NPL == 4 && VEC && !REAL;
    // fp16 tiles of 8 (eight neurons per lane, one packed 16-byte load per row) and
    // real-valued tiles of 8: the same kind of assembly dispatch (som_tree8.h). These
    // sweeps are bound by instruction issue (fp16 64x64: 112.5 -> 107.2 ms, 1024x1024:
    // 544 -> 525 ms; real-valued rows over fp16 -4 to -5%, over fp32 -1 to -2%); the fp32
    // sweep of binary rows, bound by its vector-memory path, keeps the C++ dispatch (the
    // block made it 1-4% slower).
    constexpr bool T8 = sizeof(E) == 2 && TA == 8 && NPL == 8 && VEC && !REAL;
    constexpr bool T8R = TA == 8 && NPL == 8 && VEC && REAL;
    // One vector load per row and lane (tiles of 16, and fp16 tiles of 8): the row address
    // is one vector multiply-add from the lane's own strip start (fp16: -1% sweep time).
    constexpr bool LROW = T16 || (sizeof(E) == 2 && TA == 8 && NPL == 8 && VEC);
    const char *lrow = nullptr;
    unsigned pitch = 0;
    if constexpr (LROW) {
        const int g = base + lg;
        lrow = reinterpret_cast<const char *>(W + (g < Mi ? g : Mi - G));
        pitch = (unsigned)Mi * (unsigned)sizeof(E);
        asm volatile("" : "+v"(pitch));
    }

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
            if constexpr (LROW) {
                const unsigned idc = id < vmax ? id : vmax;
                seg.v[0] = *reinterpret_cast<const typename Seg::vec *>(lrow + (uint64_t)idc * pitch);
                return;
            }
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
            if constexpr (T16) {
                const float w[4] = {seg.v[0][0], seg.v[0][1], seg.v[0][2], seg.v[0][3]};
                SOM_T16_DISPATCH(acc, w, mask);
            } else if constexpr (T8R && sizeof(E) == 4) {
                const float w[8] = {seg.v[0][0], seg.v[0][1], seg.v[0][2], seg.v[0][3],
                                    seg.v[1][0], seg.v[1][1], seg.v[1][2], seg.v[1][3]};
                SOM_T8_DISPATCH32R(acc, w, xv, mask);
            } else if constexpr (T8R) {
                const unsigned *dw = reinterpret_cast<const unsigned *>(&seg.v[0]);
                const unsigned d[4] = {dw[0], dw[1], dw[2], dw[3]};
                SOM_T8_DISPATCH16R(acc, d, xv, mask);
            } else if constexpr (T8) {
                const unsigned *dw = reinterpret_cast<const unsigned *>(&seg.v[0]);
                const unsigned d[4] = {dw[0], dw[1], dw[2], dw[3]};
                SOM_T8_DISPATCH16(acc, d, mask);
            } else if constexpr (sizeof(E) == 2 && VEC) {
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

}  // namespace

// --------------------------------------------------------------- launcher

template <typename E, int TA, int NPL, bool TOP2, bool REAL>
static void sweep_ta(bool vec, dim3 grid, int64_t group_tiles, hipStream_t st, const E *W, const double *norms,
                     int64_t M, int64_t N, int64_t V, int64_t nnz, const uint2 *plan, const int2 *tiles, int64_t nt,
                     const SweepOut &o, const float *vals)
{
    // Packed fp16 rows take half the registers: eight rows in flight still fit 128 VGPRs
    // (six for real-valued rows, whose per-entry values take scalar registers).
    // Tiles of 16 with fp32 rows of four neurons per lane: four registers a row, eight in
    // flight (tiles of 32 keep four: their 128 accumulators leave no room).
    constexpr int UV = (sizeof(E) == 2 && NPL == 8) ? (REAL ? 6 : 8) : (sizeof(E) == 4 && TA == 16 ? 8 : 4);
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
// From 60,000 tiles on, groups hold at least 8 tiles (two per wave): the 1024 x 1024
// map's 500,000 rows (62,500 tiles) then still span 7,800 groups, about seven rounds,
// per strip, and the sweep takes 769 ms instead of 784; 12 or 16 tiles (5,200 or
// 3,900 groups) cost 4-7%.
static int64_t sweep_group_tiles(int64_t nt)
{
    int64_t g = nt / 16384 / 4 * 4;
    if (g < 8 && nt >= 8 * 7500) g = 8;
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

}  // namespace som
