// som_tree8.h -- the sweep's per-row sample dispatch for tiles of 8 samples with eight
// neurons per lane (gfx950 assembly): packed fp16 rows, and real-valued rows over an fp32
// or fp16 codebook.
//
// A codebook row of a tile's union is added into the accumulators of every sample
// of the tile that holds the row's feature (the SpMM-tile kernel section). The plan
// word says which: an 8-bit sample mask, and, for a feature held by one sample (most
// union entries), that sample's slot in bits 24-26 with bit 31 clear. One inline
// assembly block per row does the whole dispatch on the wave-uniform plan word:
//  * one sample: a binary search on the slot (three scalar bit tests), then the
//    eight adds of that slot;
//  * several samples (bit 31 set): each half of the mask is tested at once, then
//    each bit of a non-empty half, with eight adds per set bit.
// As for tiles of 16 (som_tree16.h), one block keeps the 64 accumulators in place.
//
// Operands: acc[s][j] as [aS_J] (read and written), the plan word as [y] (scalar), a
// scratch scalar register [t], the row as [w0]..[w7] (fp32) or as four dwords of two
// halves each, [d0]..[d3] (fp16: neuron 2k is the low half of dword k), and for
// real-valued rows the samples' values as [x0]..[x7] (scalar).
#pragma once

// fp16: acc + h * 1.0 with h read as a half from the dword (exact widening, one rounding)
#define SOM_T8_MIX(S, J, D, SEL) "v_fma_mix_f32 %[a" #S "_" #J "], %[d" #D "], 1.0, %[a" #S "_" #J "] " SEL "\n"
#define SOM_T8_ADD16(S)                                                                  \
    SOM_T8_MIX(S, 0, 0, "op_sel_hi:[1,0,0]") SOM_T8_MIX(S, 1, 0, "op_sel:[1,0,0] op_sel_hi:[1,0,0]") \
    SOM_T8_MIX(S, 2, 1, "op_sel_hi:[1,0,0]") SOM_T8_MIX(S, 3, 1, "op_sel:[1,0,0] op_sel_hi:[1,0,0]") \
    SOM_T8_MIX(S, 4, 2, "op_sel_hi:[1,0,0]") SOM_T8_MIX(S, 5, 2, "op_sel:[1,0,0] op_sel_hi:[1,0,0]") \
    SOM_T8_MIX(S, 6, 3, "op_sel_hi:[1,0,0]") SOM_T8_MIX(S, 7, 3, "op_sel:[1,0,0] op_sel_hi:[1,0,0]")

// real-valued rows: acc += x_s * w with one fused multiply-add (fp32 codebook), or
// acc + h * x_s with h read as a half (fp16 codebook); the same bits as the C++ fmaf
#define SOM_T8_FMA(S, J) "v_fma_f32 %[a" #S "_" #J "], %[w" #J "], %[x" #S "], %[a" #S "_" #J "]\n"
#define SOM_T8_FMA32(S)                                                                   \
    SOM_T8_FMA(S, 0) SOM_T8_FMA(S, 1) SOM_T8_FMA(S, 2) SOM_T8_FMA(S, 3) SOM_T8_FMA(S, 4) \
        SOM_T8_FMA(S, 5) SOM_T8_FMA(S, 6) SOM_T8_FMA(S, 7)
#define SOM_T8_MIXX(S, J, D, SEL) "v_fma_mix_f32 %[a" #S "_" #J "], %[d" #D "], %[x" #S "], %[a" #S "_" #J "] " SEL "\n"
#define SOM_T8_FMA16(S)                                                                   \
    SOM_T8_MIXX(S, 0, 0, "op_sel_hi:[1,0,0]") SOM_T8_MIXX(S, 1, 0, "op_sel:[1,0,0] op_sel_hi:[1,0,0]") \
    SOM_T8_MIXX(S, 2, 1, "op_sel_hi:[1,0,0]") SOM_T8_MIXX(S, 3, 1, "op_sel:[1,0,0] op_sel_hi:[1,0,0]") \
    SOM_T8_MIXX(S, 4, 2, "op_sel_hi:[1,0,0]") SOM_T8_MIXX(S, 5, 2, "op_sel:[1,0,0] op_sel_hi:[1,0,0]") \
    SOM_T8_MIXX(S, 6, 3, "op_sel_hi:[1,0,0]") SOM_T8_MIXX(S, 7, 3, "op_sel:[1,0,0] op_sel_hi:[1,0,0]")

// One sample: the leaves of the search, each ending at the block's end.
#define SOM_T8_N1(ADD, A) ADD(A) "s_branch L%=_e\n"
#define SOM_T8_N2(ADD, A, B)                                                                  \
    "s_bitcmp1_b32 %[y], 24\n"                                                                \
    "s_cbranch_scc1 L%=_n" #B "_1\n" SOM_T8_N1(ADD, A) "L%=_n" #B "_1:\n" SOM_T8_N1(ADD, B)
#define SOM_T8_N4(ADD, A, B, C, D)                                                            \
    "s_bitcmp1_b32 %[y], 25\n"                                                                \
    "s_cbranch_scc1 L%=_n" #C "_2\n" SOM_T8_N2(ADD, A, B) "L%=_n" #C "_2:\n" SOM_T8_N2(ADD, C, D)
#define SOM_T8_N8(ADD)                                                                        \
    "s_bitcmp1_b32 %[y], 26\n"                                                                \
    "s_cbranch_scc1 L%=_n4_4\n" SOM_T8_N4(ADD, 0, 1, 2, 3) "L%=_n4_4:\n" SOM_T8_N4(ADD, 4, 5, 6, 7)

// Several samples: halves of the mask, then bits.
#define SOM_T8_BIT(ADD, S) \
    "s_bitcmp1_b32 %[y], " #S "\ns_cbranch_scc0 L%=_b" #S "\n" ADD(S) "L%=_b" #S ":\n"
#define SOM_T8_HALF(ADD, Q, MASK, A, B, C, D)                                                  \
    "s_and_b32 %[t], %[y], " #MASK "\ns_cbranch_scc0 L%=_q" #Q "\n" SOM_T8_BIT(ADD, A) SOM_T8_BIT(ADD, B) \
        SOM_T8_BIT(ADD, C) SOM_T8_BIT(ADD, D) "L%=_q" #Q ":\n"

#define SOM_T8_TEXT(ADD)                                                                      \
    "s_bitcmp1_b32 %[y], 31\n"                                                                \
    "s_cbranch_scc1 L%=_m\n" SOM_T8_N8(ADD) "L%=_m:\n" SOM_T8_HALF(ADD, 0, 0xf, 0, 1, 2, 3)   \
        SOM_T8_HALF(ADD, 1, 0xf0, 4, 5, 6, 7) "L%=_e:\n"

#define SOM_T8_ACC(ACC_, S)                                                                    \
    [a##S##_0] "+v"(ACC_[S][0]), [a##S##_1] "+v"(ACC_[S][1]), [a##S##_2] "+v"(ACC_[S][2]),    \
        [a##S##_3] "+v"(ACC_[S][3]), [a##S##_4] "+v"(ACC_[S][4]), [a##S##_5] "+v"(ACC_[S][5]), \
        [a##S##_6] "+v"(ACC_[S][6]), [a##S##_7] "+v"(ACC_[S][7])
#define SOM_T8_ACCS(ACC_)                                                                             \
    SOM_T8_ACC(ACC_, 0), SOM_T8_ACC(ACC_, 1), SOM_T8_ACC(ACC_, 2), SOM_T8_ACC(ACC_, 3),               \
        SOM_T8_ACC(ACC_, 4), SOM_T8_ACC(ACC_, 5), SOM_T8_ACC(ACC_, 6), SOM_T8_ACC(ACC_, 7)

// ACC_: float[8][8], D_: unsigned[4] (eight halves), Y_: the plan word.
#define SOM_T8_DISPATCH16(ACC_, D_, Y_)                                                             \
    do {                                                                                         \
        unsigned som_t8_scratch_;                                                                \
        asm volatile(SOM_T8_TEXT(SOM_T8_ADD16)                                                   \
                     : SOM_T8_ACCS(ACC_), [t] "=&s"(som_t8_scratch_)                             \
                     : [d0] "v"((D_)[0]), [d1] "v"((D_)[1]), [d2] "v"((D_)[2]), [d3] "v"((D_)[3]), \
                       [y] "s"(Y_)                                                               \
                     : "scc");                                                                   \
    } while (0)

#define SOM_T8_XS(X_)                                                                          \
    [x0] "s"((X_)[0]), [x1] "s"((X_)[1]), [x2] "s"((X_)[2]), [x3] "s"((X_)[3]), [x4] "s"((X_)[4]), \
        [x5] "s"((X_)[5]), [x6] "s"((X_)[6]), [x7] "s"((X_)[7])

// Real-valued rows over an fp32 codebook. ACC_: float[8][8], W_: float[8], X_: float[8]
// (the samples' values), Y_: the plan word.
#define SOM_T8_DISPATCH32R(ACC_, W_, X_, Y_)                                                     \
    do {                                                                                         \
        unsigned som_t8_scratch_;                                                                \
        asm volatile(SOM_T8_TEXT(SOM_T8_FMA32)                                                   \
                     : SOM_T8_ACCS(ACC_), [t] "=&s"(som_t8_scratch_)                             \
                     : [w0] "v"((W_)[0]), [w1] "v"((W_)[1]), [w2] "v"((W_)[2]), [w3] "v"((W_)[3]), \
                       [w4] "v"((W_)[4]), [w5] "v"((W_)[5]), [w6] "v"((W_)[6]), [w7] "v"((W_)[7]), \
                       SOM_T8_XS(X_), [y] "s"(Y_)                                                \
                     : "scc");                                                                   \
    } while (0)

// Real-valued rows over an fp16 codebook. D_: unsigned[4] (eight halves).
#define SOM_T8_DISPATCH16R(ACC_, D_, X_, Y_)                                                     \
    do {                                                                                         \
        unsigned som_t8_scratch_;                                                                \
        asm volatile(SOM_T8_TEXT(SOM_T8_FMA16)                                                   \
                     : SOM_T8_ACCS(ACC_), [t] "=&s"(som_t8_scratch_)                             \
                     : [d0] "v"((D_)[0]), [d1] "v"((D_)[1]), [d2] "v"((D_)[2]), [d3] "v"((D_)[3]), \
                       SOM_T8_XS(X_), [y] "s"(Y_)                                                \
                     : "scc");                                                                   \
    } while (0)
