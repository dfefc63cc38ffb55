// Element values of every weight format, four at a time: the dequantization
// routine shared by the standalone dequantization and by the attention
// kernel's KV-cache loads (Sec. 3.3: the same per-format dequantization
// serves weights and the KV cache).
//
// Each element's closed form (Eq. (1) of Sec. 2.2) is evaluated with exact
// float32 products and at most one rounding; see dequant.hip.
#pragma once

#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {

// the 4 elements e .. e+3 (e a multiple of 4)
template <int FMT>
__device__ __forceinline__ float4 value4(const uint8_t* __restrict__ W, int64_t off1, int64_t off2, int64_t off3,
                                        int64_t e) {
    float4 v;
    if constexpr (FMT == LW_F16) {
        const uint2 h = *reinterpret_cast<const uint2*>(W + 2 * e);
        v.x = half_bits_to_float(h.x & 0xFFFFu);
        v.y = half_bits_to_float(h.x >> 16);
        v.z = half_bits_to_float(h.y & 0xFFFFu);
        v.w = half_bits_to_float(h.y >> 16);
    } else if constexpr (FMT == LW_Q8_0) {
        const uint32_t q = *reinterpret_cast<const uint32_t*>(W + e);
        const float d = half_bits_to_float(*reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 5)));
        v.x = sbyte<0>(q) * d;
        v.y = sbyte<1>(q) * d;
        v.z = sbyte<2>(q) * d;
        v.w = sbyte<3>(q) * d;
    } else if constexpr (FMT == LW_Q1_0) {
        // bit (e mod 8) of byte e/8; the 4 bits of e..e+3 share one byte
        const uint32_t b = (uint32_t)W[e >> 3] >> (e & 4);
        const float d = half_bits_to_float(*reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 7)));
        v.x = (b & 1u) ? d : -d;
        v.y = (b & 2u) ? d : -d;
        v.z = (b & 4u) ? d : -d;
        v.w = (b & 8u) ? d : -d;
    } else if constexpr (FMT == LW_MXFP4) {
        // e2m1 codes in the Q4 nibble order; one e8m0 exponent per group
        const int64_t g = e >> 5;
        const int i0 = (int)(e & 31);
        uint32_t b = *reinterpret_cast<const uint32_t*>(W + 16 * g + (i0 & 15));
        b = (i0 < 16) ? (b & 0x0F0F0F0Fu) : ((b >> 4) & 0x0F0F0F0Fu);
        const float s = e8m0_to_float(W[off1 + g]);
        // binary16 e2m1 * 2^-14, times 2^14 (exact), times the scale (exact
        // unless the product leaves binary32's range)
        v.x = half_bits_to_float(e2m1_half_bits(b & 15u)) * 16384.0f * s;
        v.y = half_bits_to_float(e2m1_half_bits((b >> 8) & 15u)) * 16384.0f * s;
        v.z = half_bits_to_float(e2m1_half_bits((b >> 16) & 15u)) * 16384.0f * s;
        v.w = half_bits_to_float(e2m1_half_bits(b >> 24)) * 16384.0f * s;
    } else if constexpr (FMT == LW_Q2_K) {
        // four 2-bit codes of byte e/4; the sub-block's {scale, min} byte
        const uint32_t b = W[e >> 2];
        const uint32_t scm = W[off1 + (e >> 4)];
        const uint32_t dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * (e >> 8));
        const float ds = half_bits_to_float(dd & 0xFFFFu) * (float)(scm & 15u);  // exact
        const float dm = half_bits_to_float(dd >> 16) * (float)(scm >> 4);       // exact
        v.x = __builtin_fmaf(ds, (float)(b & 3u), -dm);                          // one rounding
        v.y = __builtin_fmaf(ds, (float)((b >> 2) & 3u), -dm);
        v.z = __builtin_fmaf(ds, (float)((b >> 4) & 3u), -dm);
        v.w = __builtin_fmaf(ds, (float)(b >> 6), -dm);
    } else {
        // Q4 code plane: group g = e/32 owns bytes [16g, 16g+16); byte i
        // holds element 32g+i (low nibble) and 32g+i+16 (high nibble).
        const int64_t g = e >> 5;
        const int i0 = (int)(e & 31);  // multiple of 4
        uint32_t b = *reinterpret_cast<const uint32_t*>(W + 16 * g + (i0 & 15));
        b = (i0 < 16) ? (b & 0x0F0F0F0Fu) : ((b >> 4) & 0x0F0F0F0Fu);
        b = opaque(b);
        if constexpr (FMT == LW_Q4_0) {
            const float d = half_bits_to_float(*reinterpret_cast<const uint16_t*>(W + off1 + 2 * g));
            v.x = (ubyte<0>(b) - 8.0f) * d;
            v.y = (ubyte<1>(b) - 8.0f) * d;
            v.z = (ubyte<2>(b) - 8.0f) * d;
            v.w = (ubyte<3>(b) - 8.0f) * d;
        } else if constexpr (FMT == LW_Q4_1) {
            const uint32_t dm = *reinterpret_cast<const uint32_t*>(W + off1 + 4 * g);
            const float d = half_bits_to_float(dm & 0xFFFFu), m = half_bits_to_float(dm >> 16);
            v.x = __builtin_fmaf(ubyte<0>(b), d, m);  // exact product, one rounding
            v.y = __builtin_fmaf(ubyte<1>(b), d, m);
            v.z = __builtin_fmaf(ubyte<2>(b), d, m);
            v.w = __builtin_fmaf(ubyte<3>(b), d, m);
        } else if constexpr (FMT == LW_Q5_0 || FMT == LW_Q5_1 || FMT == LW_Q5_K) {
            // fifth bits of e..e+3: bits (e mod 8) .. (e mod 8) + 3 of byte e/8
            const uint32_t h = ((uint32_t)W[off1 + (e >> 3)] >> (e & 4)) & 15u;
            const float q0 = (float)(((b >> 0) & 0xFFu) | ((h & 1u) << 4)), q1 = (float)(((b >> 8) & 0xFFu) | ((h & 2u) << 3));
            const float q2 = (float)(((b >> 16) & 0xFFu) | ((h & 4u) << 2)), q3 = (float)(((b >> 24) & 0xFFu) | ((h & 8u) << 1));
            if constexpr (FMT == LW_Q5_0) {
                const float d = half_bits_to_float(*reinterpret_cast<const uint16_t*>(W + off2 + 2 * g));
                v.x = (q0 - 16.0f) * d;  // exact
                v.y = (q1 - 16.0f) * d;
                v.z = (q2 - 16.0f) * d;
                v.w = (q3 - 16.0f) * d;
            } else if constexpr (FMT == LW_Q5_1) {
                const uint32_t dm = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * g);
                const float d = half_bits_to_float(dm & 0xFFFFu), m = half_bits_to_float(dm >> 16);
                v.x = __builtin_fmaf(q0, d, m);  // exact product, one rounding
                v.y = __builtin_fmaf(q1, d, m);
                v.z = __builtin_fmaf(q2, d, m);
                v.w = __builtin_fmaf(q3, d, m);
            } else {
                const int64_t S = e >> 8;
                const int j = (int)(g & 7);
                const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off2 + 12 * S);
                const uint64_t lo = (uint64_t)rec[0] | ((uint64_t)rec[1] << 32);
                const uint64_t hi = (uint64_t)rec[1] | ((uint64_t)rec[2] << 32);
                const uint32_t dd = *reinterpret_cast<const uint32_t*>(W + off3 + 4 * S);
                const float ds = half_bits_to_float(dd & 0xFFFFu) * (float)((uint32_t)(lo >> (6 * j)) & 63u);
                const float dm = half_bits_to_float(dd >> 16) * (float)((uint32_t)(hi >> (16 + 6 * j)) & 63u);
                v.x = __builtin_fmaf(ds, q0, -dm);  // exact products, one rounding
                v.y = __builtin_fmaf(ds, q1, -dm);
                v.z = __builtin_fmaf(ds, q2, -dm);
                v.w = __builtin_fmaf(ds, q3, -dm);
            }
        } else if constexpr (FMT == LW_Q6_K) {
            // high two bits of e..e+3: byte e/4 of plane 1; int8 scale per 16
            const uint32_t h = W[off1 + (e >> 2)];
            const float sc = (float)(int32_t)(int8_t)W[off2 + (e >> 4)];
            const float ds = half_bits_to_float(*reinterpret_cast<const uint16_t*>(W + off3 + 2 * (e >> 8))) * sc;
            v.x = ds * (float)((int)(((b >> 0) & 0xFFu) | ((h & 3u) << 4)) - 32);  // exact (<= 23 bits)
            v.y = ds * (float)((int)(((b >> 8) & 0xFFu) | ((h & 12u) << 2)) - 32);
            v.z = ds * (float)((int)(((b >> 16) & 0xFFu) | (h & 48u)) - 32);
            v.w = ds * (float)((int)(((b >> 24) & 0xFFu) | ((h & 192u) >> 2)) - 32);
        } else {
            const int64_t S = e >> 8;
            const int j = (int)(g & 7);
            const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * S);
            const uint64_t lo = (uint64_t)rec[0] | ((uint64_t)rec[1] << 32);  // bits 0..63
            const uint64_t hi = (uint64_t)rec[1] | ((uint64_t)rec[2] << 32);  // bits 32..95
            const uint32_t sc = (uint32_t)(lo >> (6 * j)) & 63u;
            const uint32_t m = (uint32_t)(hi >> (16 + 6 * j)) & 63u;
            const uint32_t dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * S);
            const float ds = half_bits_to_float(dd & 0xFFFFu) * (float)sc;  // exact
            const float dm = half_bits_to_float(dd >> 16) * (float)m;       // exact
            v.x = __builtin_fmaf(ds, ubyte<0>(b), -dm);                    // one rounding
            v.y = __builtin_fmaf(ds, ubyte<1>(b), -dm);
            v.z = __builtin_fmaf(ds, ubyte<2>(b), -dm);
            v.w = __builtin_fmaf(ds, ubyte<3>(b), -dm);
        }
    }
    return v;
}

}  // namespace lw
