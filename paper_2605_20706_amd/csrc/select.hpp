// Kernel selection from a swept table (the tunable kernel library of Sec. 3.2,
// whose gain comes from sweeping configurations per shape).
//
// A candidate is one launch configuration the library can run: the LDS
// single-token kernel, one of a fixed set of register-kernel instantiations,
// or one of the matrix-core families. The table (select_table.inc, generated
// from the committed sweep results) maps (format, n_tok, K, M) to the fastest
// candidate measured at that shape; a call whose shape has a table entry at
// the same format, token count and K and a row count within a factor of two
// takes that entry's candidate, every other call the built-in rules.
#pragma once

#include <stdint.h>

namespace lw {

enum Cand : int {
    kCandDefault = 0,  // the built-in rules
    kCandLds = 1,      // LDS-activation single-token kernel (gemv1_kernel)
    // register-activation kernel gemv1r_kernel<FMT, NTK, CPW, WPR, G, DR> at
    // CAP workgroups per compute unit; each takes one K / 2048 (chunk count)
    kCandReg1_1x1_G8_D2_C2 = 10,  // 1 token, 1 chunk
    kCandReg1_1x1_G4_D2_C4 = 11,
    kCandReg1_1x1_G8_D3_C2 = 12,
    kCandReg1_2x1_G8_D2_C2 = 13,  // 1 token, 2 chunks: both chunks in one wave
    kCandReg1_1x2_G4_D2_C2 = 14,  //                    one chunk per wave, two waves per row
    kCandReg1_1x2_G8_D2_C1 = 15,
    kCandReg1_2x1_G8_D3_C2 = 16,
    kCandReg1_2x1_G4_D2_C4 = 17,
    kCandReg1_1x7_G2_D2_C1 = 18,  // 1 token, 7 chunks over 7 waves
    kCandReg1_1x7_G1_D2_C2 = 19,
    kCandReg1_1x7_G2_D3_C1 = 20,
    kCandReg2_1x1_G8_D2_C2 = 21,  // 2 tokens
    kCandReg2_1x2_G4_D2_C2 = 22,
    kCandReg2_1x4_G2_D2_C1 = 23,
    kCandReg2_1x7_G2_D2_C1 = 24,
    kCandReg2_1x2_G8_D2_C1 = 25,
    kCandFewtok = 30,    // few-token matrix-core kernel, activations in LDS (2..8 tokens)
    kCandMultitok = 31,  // pair-step / many-token matrix-core kernels (2..16 tokens)
    kCandPrefill = 32,   // tiled matrix-core kernel (9 or more tokens)
};

// The candidate a call of these sizes takes: LW_FORCE_CFG (a candidate
// number, for sweeps) when set, else the table entry, else kCandDefault.
int select_cand(int fmt, int64_t M, int64_t K, int64_t n_tok);

// Whether cand is a register-kernel candidate.
inline bool is_reg_cand(int cand) { return cand >= 10 && cand < 30; }

}  // namespace lw
