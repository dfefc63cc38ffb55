// Device-side helpers shared by the lw kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lw {

constexpr int kWave = 64;

// binary16 bit pattern -> float32. v_cvt_f32_f16 is exact for every pattern,
// subnormals included (half denormals are not flushed).
__device__ __forceinline__ float half_bits_to_float(uint32_t h16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h16);
}

// 16-byte load of weight data that is read exactly once: a non-temporal hint
// keeps the stream from displacing reused data (x, scales) in the caches.
__device__ __forceinline__ uint4 stream_load16(const uint8_t* p) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Hide the known-zero bits of a value from the optimiser. Without it, a mask
// such as v & 0x0F0F0F0F followed by per-byte float conversion is rewritten
// into bit-field extracts plus conversions (two operations per code); with it
// each code is one v_cvt_f32_ubyteN.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

// Byte b (0..3) of v as float: one v_cvt_f32_ubyteN.
template <int B>
__device__ __forceinline__ float ubyte(uint32_t v) {
    return (float)((v >> (8 * B)) & 0xFFu);
}

// Signed byte b of v as float.
template <int B>
__device__ __forceinline__ float sbyte(uint32_t v) {
    return (float)(int32_t)(int8_t)(uint8_t)(v >> (8 * B));
}

template <int CTRL, int ROW_MASK = 0xF, int BANK_MASK = 0xF>
__device__ __forceinline__ float dpp_move(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 ROW_MASK, BANK_MASK, false));
}

// Sum over the 64 lanes of a wave with DPP adds; the total lands in lane 63.
// row_shr 1, 2, 4, 8 leaves each 16-lane row's sum in its lane 15;
// row_bcast:15 adds row 0 into row 1 and row 2 into row 3; row_bcast:31 adds
// the first half (lane 31) into rows 2 and 3.
__device__ __forceinline__ float wave_sum_to_lane63(float v) {
    v += dpp_move<0x111>(v);
    v += dpp_move<0x112>(v);
    v += dpp_move<0x114>(v);
    v += dpp_move<0x118>(v);
    v += dpp_move<0x142, 0xA>(v);
    v += dpp_move<0x143, 0xC>(v);
    return v;
}

// 2^(E - 127) for an e8m0 exponent byte E, as float32: E = 0 is the
// subnormal 2^-127, E = 255 NaN.
__device__ __forceinline__ float e8m0_to_float(uint32_t E) {
    const uint32_t b = E == 0 ? 0x00400000u : (E == 255 ? 0x7FC00000u : (E << 23));
    return __builtin_bit_cast(float, b);
}

// A 4-bit e2m1 code in bits 0-3 of a 16-bit half made the binary16 of
// e2m1 * 2^-14: its magnitude bits to bits 9-11 (exponent bits 10-11 and the
// top mantissa bit), its sign to bit 15 (exact for every code; e = 0 lands
// in the binary16 subnormals).
__device__ __forceinline__ uint32_t e2m1_half_bits(uint32_t c) { return ((c & 7u) << 9) | ((c & 8u) << 12); }

// Four bits at positions 4-7 of g moved to bit 4 of each byte (the fifth bit
// of four 5-bit codes held one per byte): one multiply, whose four shifted
// copies of g do not overlap.
__device__ __forceinline__ uint32_t spread4(uint32_t g) { return (g * 0x00204081u) & 0x10101010u; }

// Four 2-bit fields (bits 0-7 of g) to bits 4-5 (spread2_hi) or 0-1
// (spread2_lo) of the four bytes: two shift-or-mask steps, no carries.
__device__ __forceinline__ uint32_t spread2_hi(uint32_t g) {
    const uint32_t u = ((g << 4) | (g << 16)) & 0x00F000F0u;  // fields 0, 1 at bits 4-7; 2, 3 at 20-23
    return (u | (u << 6)) & 0x30303030u;
}
__device__ __forceinline__ uint32_t spread2_lo(uint32_t g) {
    const uint32_t u = (g | (g << 12)) & 0x000F000Fu;  // fields 0, 1 at bits 0-3; 2, 3 at 16-19
    return (u | (u << 6)) & 0x03030303u;
}

// Four 1-bit codes (bits 0-3 of b4: 1 for +1, 0 for -1) -> their bfloat16
// values as two pairs (p0: codes 0, 1; p1: codes 2, 3). One multiply moves
// bit i to bit 7 of byte i (the shifted copies do not overlap); those bits
// clear the sign of the high bytes 0xBF; byte permutations pair the high
// bytes with the low byte 0x80 of +-1.
__device__ __forceinline__ void sign_pairs(uint32_t b4, uint32_t* p0, uint32_t* p1) {
    const uint32_t hi = 0xBFBFBFBFu ^ (((b4 << 7) * 0x00204081u) & 0x80808080u);
    *p0 = __builtin_amdgcn_perm(hi, 0x80808080u, 0x05010400u);
    *p1 = __builtin_amdgcn_perm(hi, 0x80808080u, 0x07030602u);
}

// Four e2m1 codes, one per byte (idx: the magnitude bits; sgn: the sign bits,
// at bit 7 of each byte) -> their four bfloat16 values as two pairs (p0:
// bytes 0, 1; p1: bytes 2, 3). Two 8-entry byte tables indexed by the
// magnitude give the high bytes (00 3F 3F 3F 40 40 40 40) and the low bytes
// (00 00 80 C0 00 40 80 C0) of 0, 0.5, 1, 1.5, 2, 3, 4, 6; the sign goes to
// bit 7 of the high byte; two more byte permutations interleave low and high
// bytes. Exact for every code.
__device__ __forceinline__ void fp4_pairs(uint32_t idx, uint32_t sgn, uint32_t* p0, uint32_t* p1) {
    const uint32_t hi = __builtin_amdgcn_perm(0x40404040u, 0x3F3F3F00u, idx) | sgn;
    const uint32_t lo = __builtin_amdgcn_perm(0xC0804000u, 0xC0800000u, idx);
    *p0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
    *p1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

}  // namespace lw
