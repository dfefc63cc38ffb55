// Device helpers shared by the matrix-core kernels of the 4-bit formats
// (gfx950, v_mfma_f32_16x16x32_bf16, wave64).
//
// Operand layout of v_mfma_f32_16x16x32_bf16 (D[16x16] += A[16x32] . B[32x16]):
// lane l = 16 g + n (g = l / 16, n = l % 16) supplies A[n][8g .. 8g+7] and
// B[8g .. 8g+7][n], and receives D[4g + v][n], v = 0..3.
//
// Within one 32-element block the contraction order is free, so lane group g
// takes the 8 elements of code word g of the block: the low nibbles of its
// bytes (block elements 4g .. 4g+3) and then their high nibbles (elements
// 16 + 4g .. 16 + 4g + 3). The activation operand is laid out in the same
// order.
#pragma once

#include "lw_device.hpp"

namespace lw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Code word w of a block -> the 8 bf16 values 128 + q in the lane-group order
// above. bf16 128 + q (q < 16) has the bit pattern 0x4300 | q, so each pair
// is one v_perm_b32 of the masked nibbles with a constant 0x43 byte.
__device__ __forceinline__ bf16x8 biased_codes(uint32_t w) {
    const uint32_t lo = opaque(w & 0x0F0F0F0Fu);
    const uint32_t hi = opaque((w >> 4) & 0x0F0F0F0Fu);
    const uint32_t k43 = 0x43434343u;
    const u32x4 v = {__builtin_amdgcn_perm(k43, lo, 0x04010400u), __builtin_amdgcn_perm(k43, lo, 0x04030402u),
                     __builtin_amdgcn_perm(k43, hi, 0x04010400u), __builtin_amdgcn_perm(k43, hi, 0x04030402u)};
    return __builtin_bit_cast(bf16x8, v);
}

// 4 x 4 transpose across the four 16-lane groups: lane (g, n) holds words
// 0..3 of block g of its row; afterwards word j of the result is word g of
// block j (two v_permlane32_swap and two v_permlane16_swap).
__device__ __forceinline__ u32x4 quad_transpose(u32x4 w) {
    const auto s02 = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
    const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    return u32x4{s01[0], s01[1], s23[0], s23[1]};
}

// Two floats -> their bf16 high parts (round to nearest even) packed in one
// word, and the bf16 of the remainders x - high (also rounded) in another.
// high + low carries 16 significant bits of each float.
__device__ __forceinline__ void split_bf16x2(float a, float b, uint32_t& hw, uint32_t& lw) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), bf16x2));
    const float ha = __builtin_bit_cast(float, h << 16), hb = __builtin_bit_cast(float, h & 0xFFFF0000u);
    hw = h;
    lw = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a - ha, b - hb}), bf16x2));
}

}  // namespace lw
