// som_tree16.h -- the sweep's per-row sample dispatch for tiles of 16 samples with
// four fp32 neurons per lane (gfx950 assembly).
//
// A codebook row of a tile's union is added into the accumulators of every sample
// of the tile that holds the row's feature (the SpMM-tile kernel section). The plan
// word says which: a 16-bit sample mask, and, for a feature held by one sample (most
// union entries), that sample's slot in bits 24-27 with bit 31 clear. One inline
// assembly block per row does the whole dispatch on the wave-uniform plan word:
//  * one sample: a binary search on the slot (four scalar bit tests), then the
//    four adds of that slot;
//  * several samples (bit 31 set): each quarter of the mask is tested at once,
//    then each bit of a non-empty quarter, with four adds per set bit.
// Written as one block so that the 64 accumulators stay where they are: the same
// branch tree in C++ makes the compiler copy accumulators between registers at
// every join.
//
// Operands: acc[s][j] as [aS_J] (read and written), the row's four values as
// [w0]..[w3], the plan word as [y] (scalar), a scratch scalar register [t].
#pragma once

#define SOM_T16_ADD4(S)                                 \
    "v_add_f32 %[a" #S "_0], %[w0], %[a" #S "_0]\n"      \
    "v_add_f32 %[a" #S "_1], %[w1], %[a" #S "_1]\n"      \
    "v_add_f32 %[a" #S "_2], %[w2], %[a" #S "_2]\n"      \
    "v_add_f32 %[a" #S "_3], %[w3], %[a" #S "_3]\n"

// One sample: the leaves of the search, each ending at the block's end.
#define SOM_T16_N1(A) SOM_T16_ADD4(A) "s_branch L%=_e\n"
#define SOM_T16_N2(A, B)                                                          \
    "s_bitcmp1_b32 %[y], 24\n"                                                    \
    "s_cbranch_scc1 L%=_n" #B "_1\n" SOM_T16_N1(A) "L%=_n" #B "_1:\n" SOM_T16_N1(B)
#define SOM_T16_N4(A, B, C, D)                                                     \
    "s_bitcmp1_b32 %[y], 25\n"                                                     \
    "s_cbranch_scc1 L%=_n" #C "_2\n" SOM_T16_N2(A, B) "L%=_n" #C "_2:\n" SOM_T16_N2(C, D)
#define SOM_T16_N8(A, B, C, D, E, F, G, H)                                         \
    "s_bitcmp1_b32 %[y], 26\n"                                                     \
    "s_cbranch_scc1 L%=_n" #E "_4\n" SOM_T16_N4(A, B, C, D) "L%=_n" #E "_4:\n"     \
    SOM_T16_N4(E, F, G, H)
#define SOM_T16_N16                                                                \
    "s_bitcmp1_b32 %[y], 27\n"                                                     \
    "s_cbranch_scc1 L%=_n8_8\n" SOM_T16_N8(0, 1, 2, 3, 4, 5, 6, 7) "L%=_n8_8:\n"   \
    SOM_T16_N8(8, 9, 10, 11, 12, 13, 14, 15)

// Several samples: quarters of the mask, then bits.
#define SOM_T16_BIT(S) \
    "s_bitcmp1_b32 %[y], " #S "\ns_cbranch_scc0 L%=_b" #S "\n" SOM_T16_ADD4(S) "L%=_b" #S ":\n"
#define SOM_T16_QUARTER(Q, MASK, A, B, C, D)                                          \
    "s_and_b32 %[t], %[y], " #MASK "\ns_cbranch_scc0 L%=_q" #Q "\n" SOM_T16_BIT(A) \
    SOM_T16_BIT(B) SOM_T16_BIT(C) SOM_T16_BIT(D) "L%=_q" #Q ":\n"

#define SOM_T16_TEXT                                                                  \
    "s_bitcmp1_b32 %[y], 31\n"                                                        \
    "s_cbranch_scc1 L%=_m\n" SOM_T16_N16 "L%=_m:\n"                                   \
    SOM_T16_QUARTER(0, 0xf, 0, 1, 2, 3) SOM_T16_QUARTER(1, 0xf0, 4, 5, 6, 7)          \
    SOM_T16_QUARTER(2, 0xf00, 8, 9, 10, 11) SOM_T16_QUARTER(3, 0xf000, 12, 13, 14, 15) \
    "L%=_e:\n"

#define SOM_T16_ACC(ACC_, S)                                                                    \
    [a##S##_0] "+v"(ACC_[S][0]), [a##S##_1] "+v"(ACC_[S][1]), [a##S##_2] "+v"(ACC_[S][2]), \
        [a##S##_3] "+v"(ACC_[S][3])

// ACC_: float[16][4], W_: float[4], Y_: the plan word.
#define SOM_T16_DISPATCH(ACC_, W_, Y_)                                                                  \
    do {                                                                                             \
        unsigned som_t16_scratch_;                                                                   \
        asm volatile(SOM_T16_TEXT                                                                    \
                     : SOM_T16_ACC(ACC_, 0), SOM_T16_ACC(ACC_, 1), SOM_T16_ACC(ACC_, 2), SOM_T16_ACC(ACC_, 3),  \
                       SOM_T16_ACC(ACC_, 4), SOM_T16_ACC(ACC_, 5), SOM_T16_ACC(ACC_, 6), SOM_T16_ACC(ACC_, 7),  \
                       SOM_T16_ACC(ACC_, 8), SOM_T16_ACC(ACC_, 9), SOM_T16_ACC(ACC_, 10), SOM_T16_ACC(ACC_, 11),\
                       SOM_T16_ACC(ACC_, 12), SOM_T16_ACC(ACC_, 13), SOM_T16_ACC(ACC_, 14),                     \
                       SOM_T16_ACC(ACC_, 15), [t] "=&s"(som_t16_scratch_)                                       \
                     : [w0] "v"((W_)[0]), [w1] "v"((W_)[1]), [w2] "v"((W_)[2]), [w3] "v"((W_)[3]),           \
                       [y] "s"(Y_)                                                                              \
                     : "scc");                                                                                   \
    } while (0)
