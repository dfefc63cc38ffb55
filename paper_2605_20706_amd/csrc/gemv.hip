// Fused dequantize x matrix-vector product (decode, n_tok <= LW_GEMV_MAX_TOK).
//
// y[t][r] = sum_k value(W, r*K + k) * x[t][k]  (Sec. 2.1: decode is a
// matrix-vector product; Sec. 3.3: the matrix-vector kernel dequantizes the
// weights directly into registers instead of tiling them through shared
// memory, and the vector is tiled and the row reduced cooperatively, Sec. 3.2).
//
// Mapping on gfx950 (wave64):
//  * A chunk is 64 lanes x 16 bytes = 1 KiB of a row's code plane: 2048
//    elements for the 4-bit formats, 1024 for Q8_0, 512 for f16. Lane l loads
//    its 16 bytes with one 128-bit load, so each wave-wide load is one
//    contiguous KiB; its block scale(s) are loaded beside it.
//  * Each wave owns R consecutive rows and walks their chunks, keeping R x NT
//    float32 partial sums per lane; at the end the 64 lanes are summed with
//    DPP adds and lane 63 stores the R x NT results.
//  * The workgroup stages its x tile once in LDS in a lane-interleaved order
//    (float4 j of lane l of chunk c at index (c*J + j)*64 + l), so every
//    128-bit LDS read of a wave is 64 consecutive float4s (no bank conflicts);
//    one x read serves the R rows of the wave.
//  * Codes become floats with one v_cvt_f32_ubyteN each (4-bit: the low and
//    high nibbles are masked in place, the high-nibble sum is scaled by 1/16
//    at the end); block scales are applied once per 32 elements in factored
//    form: Q4_0 d*(sum q*x - 8*sum x), Q4_1 d*sum q*x + m*sum x, Q4_K-style
//    d*sc*sum q*x - dmin*m*sum x,
//    with the per-group sums of x precomputed in LDS per tile.
// Accumulation is float32 throughout; only the rounding order differs from
// the plain definition.
#include <atomic>

#include "lw_device.hpp"
#include "lw_internal.hpp"
#include "select.hpp"

namespace lw {
namespace {

// names of the kernel templates, for lw_kernel_name
struct Name_gemv_kernel {
    static constexpr const char* base = "gemv_kernel";
};
struct Name_gemv1_kernel {
    static constexpr const char* base = "gemv1_kernel";
};
struct Name_gemv1r_kernel {
    static constexpr const char* base = "gemv1r_kernel";
};

constexpr int64_t kLdsBytes = 64 * 1024;      // LDS budget of a workgroup (x tile + group sums)
constexpr int64_t kRegLdsBytes = 128 * 1024;  // of a register-kernel workgroup (one per compute unit or two)

// Device view of the rows of NS matrices that share the same activations as
// one row space (lw_matvec_multi): segment i holds global rows [start[i],
// start[i] + M[i]); its plane offsets, weights and output are its own.
// Unused segments start past every row.
template <int NS>
__device__ __forceinline__ int seg_of(const RowSegs<NS>& sg, int64_t row) {
    int i = 0;
#pragma unroll
    for (int k = 1; k < NS; ++k)
        if (row >= sg.start[k]) i = k;
    return i;
}

template <int FMT>
struct Traits;

template <>
struct Traits<LW_F16> {
    static constexpr int EPL = 8;  // elements per lane per chunk
    static constexpr bool kGroupSums = false;
    struct Packet {
        uint4 c;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t, int64_t, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + 2 * e);
        return p;
    }
    // Byte offsets (wave-uniform, 32-bit: the kernel using them is chosen
    // only for planes below 4 GiB) of chunk c (512 elements) of row `row` in
    // each plane, and the packet of lane la at those offsets.
    struct Base {
        uint32_t c;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) { return {row * (2u * K) + 1024u * c}; }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t*, const uint8_t*, const Base& b, uint32_t la,
                                     const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float, int) {
        float s = 0.f;
        s = __builtin_fmaf(half_bits_to_float(p.c.x & 0xFFFFu), xv[0].x, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.x >> 16), xv[0].y, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.y & 0xFFFFu), xv[0].z, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.y >> 16), xv[0].w, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.z & 0xFFFFu), xv[1].x, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.z >> 16), xv[1].y, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.w & 0xFFFFu), xv[1].z, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.w >> 16), xv[1].w, s);
        return s;
    }
};

template <>
struct Traits<LW_Q8_0> {
    static constexpr int EPL = 16;
    static constexpr bool kGroupSums = false;
    struct Packet {
        uint4 c;
        uint32_t d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + e);
        p.d = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 5));
        return p;
    }
    struct Base {
        uint32_t c, d;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 1024 elements
        return {row * K + 1024u * c, row * (K / 16u) + 64u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t*, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.d = *reinterpret_cast<const uint16_t*>(P1 + b.d + 2u * (la >> 1));
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float, int) {
        const uint32_t w[4] = {p.c.x, p.c.y, p.c.z, p.c.w};
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            s0 = __builtin_fmaf(sbyte<0>(w[i]), xv[i].x, s0);
            s1 = __builtin_fmaf(sbyte<1>(w[i]), xv[i].y, s1);
            s0 = __builtin_fmaf(sbyte<2>(w[i]), xv[i].z, s0);
            s1 = __builtin_fmaf(sbyte<3>(w[i]), xv[i].w, s1);
        }
        return half_bits_to_float(p.d) * (s0 + s1);
    }
};

// Half h (0: bits 0..15, 1: bits 16..31) of v as a binary16 value, widened.
template <int H>
__device__ __forceinline__ float half_of(uint32_t v) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(H ? (v >> 16) : (v & 0xFFFFu)));
}

// Sum over the lane's 32 elements of q * x for 4-bit codes. A 4-bit code
// masked into the low bits of a 16-bit half is the binary16 subnormal
// q * 2^-24 (exactly); a high nibble masked in place reads as 16q * 2^-24.
// Each product then takes one v_fma_mix_f32 (binary16 x float32, fused, the
// 16-bit operand picked from its half by op_sel) and needs no conversion
// instruction; the powers of two are undone once at the end (exact).
__device__ __forceinline__ float nibble_dot(const uint4& c, const float4* xv) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    float lo_s = 0.f, hi_s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t l02 = opaque(w[i] & 0x000F000Fu);         // elements 4i, 4i+2
        const uint32_t h02 = opaque(w[i] & 0x00F000F0u);         // 16+4i, 16+4i+2 (times 16)
        const uint32_t l13 = opaque((w[i] >> 8) & 0x000F000Fu);  // 4i+1, 4i+3
        const uint32_t h13 = opaque((w[i] >> 8) & 0x00F000F0u);  // 16+4i+1, 16+4i+3 (times 16)
        lo_s = __builtin_fmaf(half_of<0>(l02), xv[i].x, lo_s);
        lo_s = __builtin_fmaf(half_of<1>(l02), xv[i].z, lo_s);
        lo_s = __builtin_fmaf(half_of<0>(l13), xv[i].y, lo_s);
        lo_s = __builtin_fmaf(half_of<1>(l13), xv[i].w, lo_s);
        hi_s = __builtin_fmaf(half_of<0>(h02), xv[4 + i].x, hi_s);
        hi_s = __builtin_fmaf(half_of<1>(h02), xv[4 + i].z, hi_s);
        hi_s = __builtin_fmaf(half_of<0>(h13), xv[4 + i].y, hi_s);
        hi_s = __builtin_fmaf(half_of<1>(h13), xv[4 + i].w, hi_s);
    }
    return __builtin_fmaf(hi_s, 1048576.0f, lo_s * 16777216.0f);  // 2^20 = 2^24 / 16, 2^24
}

template <>
struct Traits<LW_Q4_0> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.d = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 5));
        return p;
    }
    struct Base {
        uint32_t c, d;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 2048 elements
        return {row * (K / 2u) + 1024u * c, row * (K / 16u) + 128u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t*, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.d = *reinterpret_cast<const uint16_t*>(P1 + b.d + 2u * la);
        return p;
    }
    // d * (sum q*x - 8 * sum x)
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        return half_bits_to_float(p.d) * __builtin_fmaf(-8.0f, sx, nibble_dot(p.c, xv));
    }
};

// Q4_1: Q4_0's codes with a {binary16 d, binary16 m} pair per group.
template <>
struct Traits<LW_Q4_1> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t dm;  // d in bits 0..15, m in bits 16..31
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.dm = *reinterpret_cast<const uint32_t*>(W + off1 + 4 * (e >> 5));
        return p;
    }
    struct Base {
        uint32_t c, dm;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 2048 elements
        return {row * (K / 2u) + 1024u * c, row * (K / 8u) + 256u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t*, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.dm = *reinterpret_cast<const uint32_t*>(P1 + b.dm + 4u * la);
        return p;
    }
    // d * sum q*x + m * sum x
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        return __builtin_fmaf(half_bits_to_float(p.dm >> 16), sx,
                              half_bits_to_float(p.dm & 0xFFFFu) * nibble_dot(p.c, xv));
    }
};

// Sum over the lane's 32 elements of b * x for 1-bit codes b. A bit masked
// into bit 0 of a 16-bit half is the binary16 subnormal b * 2^-24 (exact), so
// as for the 4-bit codes each product is one v_fma_mix_f32 with no
// conversion; bit i and bit 16 + i (elements i and 16 + i) come out of the
// word with one shift and one mask.
__device__ __forceinline__ float bit_dot(uint32_t w, const float4* xv) {
    float lo_s = 0.f, hi_s = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const uint32_t m = opaque((w >> i) & 0x00010001u);
        const float4& xl = xv[i >> 2];
        const float4& xh = xv[4 + (i >> 2)];
        const int c = i & 3;
        lo_s = __builtin_fmaf(half_of<0>(m), c == 0 ? xl.x : c == 1 ? xl.y : c == 2 ? xl.z : xl.w, lo_s);
        hi_s = __builtin_fmaf(half_of<1>(m), c == 0 ? xh.x : c == 1 ? xh.y : c == 2 ? xh.z : xh.w, hi_s);
    }
    return (lo_s + hi_s) * 16777216.0f;  // 2^24
}

// One AND per bit pair for the 1-bit format. A single set bit i < 12 of a
// binary16 half is exactly 2^(i - 24) (bits 0..9 subnormal, bits 10 and 11
// the lowest exponent bits); bits 12..15, shifted down by 4, are bits 8..11.
// So with the lane's x pre-multiplied by 2^-s(e), s(e) = e mod 16 below 12
// and e mod 16 - 4 from 12 (q1_prescale, exact: powers of two), the masked
// bit times the pre-scaled x is b * x * 2^-24, the same product bit_dot
// forms. 16 ANDs and one shift per 32 bits instead of 16 shifts and 16 ANDs.
__device__ __forceinline__ int q1_shift(int e) {
    const int i = e & 15;
    return i < 12 ? i : i - 4;
}

__device__ __forceinline__ void q1_prescale(float4* xv) {  // the lane's 8 float4 (32 elements)
#pragma unroll
    for (int j4 = 0; j4 < 8; ++j4) {
        xv[j4].x = __builtin_ldexpf(xv[j4].x, -q1_shift(4 * j4 + 0));
        xv[j4].y = __builtin_ldexpf(xv[j4].y, -q1_shift(4 * j4 + 1));
        xv[j4].z = __builtin_ldexpf(xv[j4].z, -q1_shift(4 * j4 + 2));
        xv[j4].w = __builtin_ldexpf(xv[j4].w, -q1_shift(4 * j4 + 3));
    }
}

// The mask of bit pair i (elements i and 16 + i) of w, w4 = w >> 4.
__device__ __forceinline__ uint32_t q1_mask(uint32_t w, uint32_t w4, int i) {
    return opaque((i < 12 ? w : w4) & (0x00010001u << q1_shift(i)));
}

// bit_dot over pre-scaled x (q1_prescale)
__device__ __forceinline__ float bit_dot_pre(uint32_t w, const float4* xv) {
    float lo_s = 0.f, hi_s = 0.f;
    const uint32_t w4 = w >> 4;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const uint32_t m = q1_mask(w, w4, i);
        const float4& xl = xv[i >> 2];
        const float4& xh = xv[4 + (i >> 2)];
        const int c = i & 3;
        lo_s = __builtin_fmaf(half_of<0>(m), c == 0 ? xl.x : c == 1 ? xl.y : c == 2 ? xl.z : xl.w, lo_s);
        hi_s = __builtin_fmaf(half_of<1>(m), c == 0 ? xh.x : c == 1 ? xh.y : c == 2 ? xh.z : xh.w, hi_s);
    }
    return (lo_s + hi_s) * 16777216.0f;  // 2^24
}

// q1_0 (Sec. 2.2: one bit per weight, one binary16 scale per 128): a lane
// holds 32 consecutive bits (one 32-bit word; a wave-wide load is 256
// contiguous bytes) and its block's scale, shared by four lanes.
template <>
struct Traits<LW_Q1_0> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint32_t b;
        uint32_t d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t, int64_t = 0) {
        Packet p;
        p.b = *reinterpret_cast<const uint32_t*>(W + (e >> 3));
        p.d = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 7));
        return p;
    }
    struct Base {
        uint32_t c, d;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 2048 elements
        return {row * (K / 8u) + 256u * c, row * (K / 64u) + 32u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t*, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.b = *reinterpret_cast<const uint32_t*>(W + b.c + 4u * la);
        p.d = *reinterpret_cast<const uint16_t*>(P1 + b.d + 2u * (la >> 2));
        return p;
    }
    // sum (2b - 1) * d * x = d * (2 * sum b*x - sum x)
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        return half_bits_to_float(p.d) * __builtin_fmaf(2.0f, bit_dot(p.b, xv), -sx);
    }
    // the same over x pre-scaled by q1_prescale (sx the sum of the plain x)
    __device__ static float dot_pre(const Packet& p, const float4* xv, float sx) {
        return half_bits_to_float(p.d) * __builtin_fmaf(2.0f, bit_dot_pre(p.b, xv), -sx);
    }
};

template <>
struct Traits<LW_Q4_K> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t r0, r1, r2, dd;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * (e >> 8));
        p.r0 = rec[0];
        p.r1 = rec[1];
        p.r2 = rec[2];
        p.dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * (e >> 8));
        return p;
    }
    struct Base {
        uint32_t c, rec, dd;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 2048 elements = 8 super-blocks
        return {row * (K / 2u) + 1024u * c, row * (12u * (K / 256u)) + 96u * c, row * (4u * (K / 256u)) + 32u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(P1 + b.rec + 12u * (la >> 3));
        p.r0 = rec[0];
        p.r1 = rec[1];
        p.r2 = rec[2];
        p.dd = *reinterpret_cast<const uint32_t*>(P2 + b.dd + 4u * (la >> 3));
        return p;
    }
    // d*sc_j * sum q*x - dmin*m_j * sum x; j is the lane's sub-block (0..7).
    // The 6-bit fields are cut out of the 96-bit record {r2:r1:r0} with 32-bit
    // funnel shifts (v_alignbit_b32): no 64-bit register pairs, so the loaded
    // words are used where they land.
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int j) {
        const uint32_t ts = 6u * (uint32_t)j;         // sc_j at bit ts (0..42)
        const uint32_t tm = 16u + 6u * (uint32_t)j;   // m_j at bit 32 + tm (tm 16..58)
        const bool sl = ts < 32u, ml = tm < 32u;  // field starts in the lower word of the pair
        const uint32_t sc_w = __builtin_amdgcn_alignbit(sl ? p.r1 : 0u, sl ? p.r0 : p.r1, ts & 31u);
        const uint32_t m_w = __builtin_amdgcn_alignbit(ml ? p.r2 : 0u, ml ? p.r1 : p.r2, tm & 31u);
        const float sc = (float)(sc_w & 63u);
        const float m = (float)(m_w & 63u);
        const float ds = half_bits_to_float(p.dd & 0xFFFFu) * sc;
        const float dm = half_bits_to_float(p.dd >> 16) * m;
        return __builtin_fmaf(ds, nibble_dot(p.c, xv), -dm * sx);
    }
};

// ---- 5-bit, 6-bit and 2-bit formats ------------------------------------
// Each lane holds one 32-element group, as for the 4-bit formats: the low
// four bits of 5- and 6-bit codes come from the Q4 nibble plane, the high
// bits from a plane of their own; every product is a v_fma_mix_f32 on a code
// field masked into a binary16 subnormal.

// 8-byte load of weight data read once (non-temporal).
__device__ __forceinline__ uint2 stream_load8(const uint8_t* p) {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
    return make_uint2(v.x, v.y);
}

// sum over the lane's 32 elements of q*x for the low nibbles, split into
// elements 0..15 (sa) and 16..31 (sb), each in true units
__device__ __forceinline__ void nibble_dot2(const uint4& c, const float4* xv, float& sa, float& sb) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    float lo_s = 0.f, hi_s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t l02 = opaque(w[i] & 0x000F000Fu);
        const uint32_t h02 = opaque(w[i] & 0x00F000F0u);
        const uint32_t l13 = opaque((w[i] >> 8) & 0x000F000Fu);
        const uint32_t h13 = opaque((w[i] >> 8) & 0x00F000F0u);
        lo_s = __builtin_fmaf(half_of<0>(l02), xv[i].x, lo_s);
        lo_s = __builtin_fmaf(half_of<1>(l02), xv[i].z, lo_s);
        lo_s = __builtin_fmaf(half_of<0>(l13), xv[i].y, lo_s);
        lo_s = __builtin_fmaf(half_of<1>(l13), xv[i].w, lo_s);
        hi_s = __builtin_fmaf(half_of<0>(h02), xv[4 + i].x, hi_s);
        hi_s = __builtin_fmaf(half_of<1>(h02), xv[4 + i].z, hi_s);
        hi_s = __builtin_fmaf(half_of<0>(h13), xv[4 + i].y, hi_s);
        hi_s = __builtin_fmaf(half_of<1>(h13), xv[4 + i].w, hi_s);
    }
    sa = lo_s * 16777216.0f;  // 2^24
    sb = hi_s * 1048576.0f;   // 2^20: high nibbles read as 16q
}

// sum of q*x over 16 elements whose 2-bit fields fill one 32-bit word
// (element j at bits 2j); x4 points at their 4 float4s. (w >> 2j) masked
// with 0x00030003 holds element j in the low half and element 8 + j in the
// high half.
__device__ __forceinline__ float two_bit_dot(uint32_t w, const float4* x4) {
    float a = 0.f, b = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t m = opaque((w >> (2 * j)) & 0x00030003u);
        const float4& xl = x4[j >> 2];
        const float4& xh = x4[2 + (j >> 2)];
        const float vl = (j & 3) == 0 ? xl.x : (j & 3) == 1 ? xl.y : (j & 3) == 2 ? xl.z : xl.w;
        const float vh = (j & 3) == 0 ? xh.x : (j & 3) == 1 ? xh.y : (j & 3) == 2 ? xh.z : xh.w;
        a = __builtin_fmaf(half_of<0>(m), vl, a);
        b = __builtin_fmaf(half_of<1>(m), vh, b);
    }
    return (a + b) * 16777216.0f;  // 2^24
}

// sum of the 16 elements in 4 float4s
__device__ __forceinline__ float sum16(const float4* x4) {
    return ((x4[0].x + x4[0].y) + (x4[0].z + x4[0].w)) + ((x4[1].x + x4[1].y) + (x4[1].z + x4[1].w)) +
           (((x4[2].x + x4[2].y) + (x4[2].z + x4[2].w)) + ((x4[3].x + x4[3].y) + (x4[3].z + x4[3].w)));
}

// One AND per pair of 2-bit codes. A 2-bit field at bits 2j, 2j+1 <= 9 of a
// binary16 half lies in the mantissa, so it reads as c * 2^(2j - 24)
// exactly; fields 5..7 (bits 10..15) are shifted down by 6 first (bits
// 4..9). With the lane's x pre-multiplied by 2^-t(e) (q2_prescale: t = 2j
// for fields 0..4, 2j - 6 for 5..7, j = (e mod 16) mod 8 the field of element
// e), each masked field times its x is c * x * 2^-24, the product
// two_bit_dot forms. 9 instead of 16 mask instructions per 16 codes.
__device__ __forceinline__ int q2_shift(int e) {
    const int j = (e & 15) & 7;
    return j <= 4 ? 2 * j : 2 * j - 6;
}

__device__ __forceinline__ void q2_prescale(float4* xv) {  // the lane's 8 float4 (32 elements)
#pragma unroll
    for (int j4 = 0; j4 < 8; ++j4) {
        xv[j4].x = __builtin_ldexpf(xv[j4].x, -q2_shift(4 * j4 + 0));
        xv[j4].y = __builtin_ldexpf(xv[j4].y, -q2_shift(4 * j4 + 1));
        xv[j4].z = __builtin_ldexpf(xv[j4].z, -q2_shift(4 * j4 + 2));
        xv[j4].w = __builtin_ldexpf(xv[j4].w, -q2_shift(4 * j4 + 3));
    }
}

// two_bit_dot over x pre-scaled by q2_prescale
__device__ __forceinline__ float two_bit_dot_pre(uint32_t w, const float4* x4) {
    float a = 0.f, b = 0.f;
    const uint32_t w6 = w >> 6;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t m = opaque((j <= 4 ? w : w6) & (0x00030003u << (j <= 4 ? 2 * j : 2 * j - 6)));
        const float4& xl = x4[j >> 2];
        const float4& xh = x4[2 + (j >> 2)];
        const float vl = (j & 3) == 0 ? xl.x : (j & 3) == 1 ? xl.y : (j & 3) == 2 ? xl.z : xl.w;
        const float vh = (j & 3) == 0 ? xh.x : (j & 3) == 1 ? xh.y : (j & 3) == 2 ? xh.z : xh.w;
        a = __builtin_fmaf(half_of<0>(m), vl, a);
        b = __builtin_fmaf(half_of<1>(m), vh, b);
    }
    return (a + b) * 16777216.0f;  // 2^24
}

// The 6-bit sub-block fields of a K-quant record {r0, r1, r2} (sc_j at bit
// 6j, m_j at bit 48 + 6j), as floats.
__device__ __forceinline__ void record_fields(uint32_t r0, uint32_t r1, uint32_t r2, int j, float& sc, float& m) {
    const uint32_t ts = 6u * (uint32_t)j;
    const uint32_t tm = 16u + 6u * (uint32_t)j;
    const bool sl = ts < 32u, ml = tm < 32u;
    const uint32_t sc_w = __builtin_amdgcn_alignbit(sl ? r1 : 0u, sl ? r0 : r1, ts & 31u);
    const uint32_t m_w = __builtin_amdgcn_alignbit(ml ? r2 : 0u, ml ? r1 : r2, tm & 31u);
    sc = (float)(sc_w & 63u);
    m = (float)(m_w & 63u);
}

// Q5_0: value d * (q - 16), q = nibble + 16 * fifth bit.
template <>
struct Traits<LW_Q5_0> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t h, d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.h = *reinterpret_cast<const uint32_t*>(W + off1 + (e >> 3));
        p.d = *reinterpret_cast<const uint16_t*>(W + off2 + 2 * (e >> 5));
        return p;
    }
    struct Base {
        uint32_t c, h, d;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 2048 elements
        return {row * (K / 2u) + 1024u * c, row * (K / 8u) + 256u * c, row * (K / 16u) + 128u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.h = *reinterpret_cast<const uint32_t*>(P1 + b.h + 4u * la);
        p.d = *reinterpret_cast<const uint16_t*>(P2 + b.d + 2u * la);
        return p;
    }
    // d * (sum q*x - 16 * sum x)
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        const float q = __builtin_fmaf(16.0f, bit_dot(p.h, xv), nibble_dot(p.c, xv));
        return half_bits_to_float(p.d) * __builtin_fmaf(-16.0f, sx, q);
    }
};

// Q5_1: value d * q + m.
template <>
struct Traits<LW_Q5_1> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t h, dm;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.h = *reinterpret_cast<const uint32_t*>(W + off1 + (e >> 3));
        p.dm = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * (e >> 5));
        return p;
    }
    struct Base {
        uint32_t c, h, dm;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {
        return {row * (K / 2u) + 1024u * c, row * (K / 8u) + 256u * c, row * (K / 8u) + 256u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.h = *reinterpret_cast<const uint32_t*>(P1 + b.h + 4u * la);
        p.dm = *reinterpret_cast<const uint32_t*>(P2 + b.dm + 4u * la);
        return p;
    }
    // d * sum q*x + m * sum x
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        const float q = __builtin_fmaf(16.0f, bit_dot(p.h, xv), nibble_dot(p.c, xv));
        return __builtin_fmaf(half_bits_to_float(p.dm >> 16), sx, half_bits_to_float(p.dm & 0xFFFFu) * q);
    }
};

// Q5_K-style: value d*sc_j*q - dmin*m_j with 5-bit q.
template <>
struct Traits<LW_Q5_K> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t h, r0, r1, r2, dd;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2, int64_t off3 = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.h = *reinterpret_cast<const uint32_t*>(W + off1 + (e >> 3));
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off2 + 12 * (e >> 8));
        p.r0 = rec[0];
        p.r1 = rec[1];
        p.r2 = rec[2];
        p.dd = *reinterpret_cast<const uint32_t*>(W + off3 + 4 * (e >> 8));
        return p;
    }
    struct Base {
        uint32_t c, h, rec, dd;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {
        return {row * (K / 2u) + 1024u * c, row * (K / 8u) + 256u * c, row * (12u * (K / 256u)) + 96u * c,
                row * (4u * (K / 256u)) + 32u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const Base& b,
                                     uint32_t la, const uint8_t* P3 = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.h = *reinterpret_cast<const uint32_t*>(P1 + b.h + 4u * la);
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(P2 + b.rec + 12u * (la >> 3));
        p.r0 = rec[0];
        p.r1 = rec[1];
        p.r2 = rec[2];
        p.dd = *reinterpret_cast<const uint32_t*>(P3 + b.dd + 4u * (la >> 3));
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int j) {
        float sc, m;
        record_fields(p.r0, p.r1, p.r2, j, sc, m);
        const float ds = half_bits_to_float(p.dd & 0xFFFFu) * sc;
        const float dm = half_bits_to_float(p.dd >> 16) * m;
        const float q = __builtin_fmaf(16.0f, bit_dot(p.h, xv), nibble_dot(p.c, xv));
        return __builtin_fmaf(ds, q, -dm * sx);
    }
};

// Q6_K-style: value d*sc_t*(q - 32), sub-blocks of 16 (a lane's group is two).
template <>
struct Traits<LW_Q6_K> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint2 h;
        uint32_t sc, d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2, int64_t off3 = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.h = *reinterpret_cast<const uint2*>(W + off1 + (e >> 2));
        p.sc = *reinterpret_cast<const uint16_t*>(W + off2 + (e >> 4));
        p.d = *reinterpret_cast<const uint16_t*>(W + off3 + 2 * (e >> 8));
        return p;
    }
    struct Base {
        uint32_t c, h, sc, d;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {
        return {row * (K / 2u) + 1024u * c, row * (K / 4u) + 512u * c, row * (K / 16u) + 128u * c,
                row * (2u * (K / 256u)) + 16u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const Base& b,
                                     uint32_t la, const uint8_t* P3 = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.h = stream_load8(P1 + b.h + 8u * la);
        p.sc = *reinterpret_cast<const uint16_t*>(P2 + b.sc + 2u * la);
        p.d = *reinterpret_cast<const uint16_t*>(P3 + b.d + 2u * (la >> 3));
        return p;
    }
    // d * sum over the two sub-blocks of sc_t * (sum q*x - 32 * sum x)
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        float la, lb;
        nibble_dot2(p.c, xv, la, lb);
        const float qa = __builtin_fmaf(16.0f, two_bit_dot(p.h.x, xv), la);
        const float qb = __builtin_fmaf(16.0f, two_bit_dot(p.h.y, xv + 4), lb);
        const float sxa = sum16(xv), sxb = sx - sxa;
        const float sca = (float)(int32_t)(int8_t)(p.sc & 0xFFu);
        const float scb = (float)(int32_t)(int8_t)(p.sc >> 8);
        const float t = sca * __builtin_fmaf(-32.0f, sxa, qa);
        return half_bits_to_float(p.d) * __builtin_fmaf(scb, __builtin_fmaf(-32.0f, sxb, qb), t);
    }
};

// Q2_K-style: value d*sc_t*q - dmin*m_t with 2-bit q, sub-blocks of 16.
template <>
struct Traits<LW_Q2_K> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint2 c;
        uint32_t scm, dd;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint2*>(W + (e >> 2));
        p.scm = *reinterpret_cast<const uint16_t*>(W + off1 + (e >> 4));
        p.dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * (e >> 8));
        return p;
    }
    struct Base {
        uint32_t c, scm, dd;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {
        return {row * (K / 4u) + 512u * c, row * (K / 16u) + 128u * c, row * (4u * (K / 256u)) + 32u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const Base& b,
                                     uint32_t la, const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load8(W + b.c + 8u * la);
        p.scm = *reinterpret_cast<const uint16_t*>(P1 + b.scm + 2u * la);
        p.dd = *reinterpret_cast<const uint32_t*>(P2 + b.dd + 4u * (la >> 3));
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        const float qa = two_bit_dot(p.c.x, xv), qb = two_bit_dot(p.c.y, xv + 4);
        const float sxa = sum16(xv), sxb = sx - sxa;
        const float d = half_bits_to_float(p.dd & 0xFFFFu), dmin = half_bits_to_float(p.dd >> 16);
        const float dsa = d * (float)(p.scm & 15u), dma = dmin * (float)((p.scm >> 4) & 15u);
        const float dsb = d * (float)((p.scm >> 8) & 15u), dmb = dmin * (float)((p.scm >> 12) & 15u);
        return __builtin_fmaf(dsa, qa, -dma * sxa) + __builtin_fmaf(dsb, qb, -dmb * sxb);
    }
    // the same over x pre-scaled by q2_prescale, sxa the sum of the plain x's
    // first 16 elements (staged once with x)
    __device__ static float dot_pre(const Packet& p, const float4* xv, float sx, float sxa) {
        const float qa = two_bit_dot_pre(p.c.x, xv), qb = two_bit_dot_pre(p.c.y, xv + 4);
        const float sxb = sx - sxa;
        const float d = half_bits_to_float(p.dd & 0xFFFFu), dmin = half_bits_to_float(p.dd >> 16);
        const float dsa = d * (float)(p.scm & 15u), dma = dmin * (float)((p.scm >> 4) & 15u);
        const float dsb = d * (float)((p.scm >> 8) & 15u), dmb = dmin * (float)((p.scm >> 12) & 15u);
        return __builtin_fmaf(dsa, qa, -dma * sxa) + __builtin_fmaf(dsb, qb, -dmb * sxb);
    }
};

// mxfp4: e2m1 codes in the Q4 nibble order and one e8m0 exponent per group.
// Each code becomes the binary16 e2m1 * 2^-14 (its magnitude bits moved to
// bits 9-11, its sign to bit 15), so every product is one v_fma_mix_f32 in
// units of 2^-14; the lane's sum is scaled by 2^14 and the block's 2^(E-127).
__device__ __forceinline__ float e2m1_dot(const uint4& c, const float4* xv) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    float lo_s = 0.f, hi_s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t v = w[i];
        const uint32_t l02 = opaque(((v & 0x00070007u) << 9) | ((v & 0x00080008u) << 12));  // elements 4i, 4i+2
        const uint32_t h02 = opaque(((v & 0x00700070u) << 5) | ((v & 0x00800080u) << 8));   // 16+4i, 16+4i+2
        const uint32_t l13 = opaque(((v & 0x07000700u) << 1) | ((v & 0x08000800u) << 4));   // 4i+1, 4i+3
        const uint32_t h13 = opaque(((v & 0x70007000u) >> 3) | (v & 0x80008000u));         // 16+4i+1, 16+4i+3
        lo_s = __builtin_fmaf(half_of<0>(l02), xv[i].x, lo_s);
        lo_s = __builtin_fmaf(half_of<1>(l02), xv[i].z, lo_s);
        lo_s = __builtin_fmaf(half_of<0>(l13), xv[i].y, lo_s);
        lo_s = __builtin_fmaf(half_of<1>(l13), xv[i].w, lo_s);
        hi_s = __builtin_fmaf(half_of<0>(h02), xv[4 + i].x, hi_s);
        hi_s = __builtin_fmaf(half_of<1>(h02), xv[4 + i].z, hi_s);
        hi_s = __builtin_fmaf(half_of<0>(h13), xv[4 + i].y, hi_s);
        hi_s = __builtin_fmaf(half_of<1>(h13), xv[4 + i].w, hi_s);
    }
    return (lo_s + hi_s) * 16384.0f;  // 2^14
}

template <>
struct Traits<LW_MXFP4> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = false;
    struct Packet {
        uint4 c;
        uint32_t E;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t, int64_t = 0) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.E = W[off1 + (e >> 5)];
        return p;
    }
    struct Base {
        uint32_t c, E;
    };
    __device__ static Base base(uint32_t row, uint32_t K, uint32_t c) {  // chunk = 2048 elements
        return {row * (K / 2u) + 1024u * c, row * (K / 32u) + 64u * c};
    }
    __device__ static Packet load_at(const uint8_t* W, const uint8_t* P1, const uint8_t*, const Base& b, uint32_t la,
                                     const uint8_t* = nullptr) {
        Packet p;
        p.c = stream_load16(W + b.c + 16u * la);
        p.E = P1[b.E + la];
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float, int) {
        return e2m1_dot(p.c, xv) * e8m0_to_float(p.E);
    }
};

// Scaled forms for the register kernel: the lane's 32 products are
// accumulated in units of 2^-24 (the value of a nibble masked into the low
// bits of a binary16 half), so no per-step rescaling is needed; the caller
// multiplies the row total by 2^24 once, after the cross-lane sum (exact:
// powers of two). sx24 is the lane's group sum of x times 2^-24.
//
// For NTK tokens at once (the masks are shared): out[t] = sum over the lane's
// 32 elements of q * x_t in units of 2^-24. xv[t] points at token t's 8 float4s.
template <int NTK>
__device__ __forceinline__ void nibble_dot24(const uint4& c, const float4* const* xv, float* out) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    float lo_s[NTK], hi_s[NTK];
#pragma unroll
    for (int t = 0; t < NTK; ++t) lo_s[t] = hi_s[t] = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t l02 = opaque(w[i] & 0x000F000Fu);
        const uint32_t h02 = opaque(w[i] & 0x00F000F0u);
        const uint32_t l13 = opaque((w[i] >> 8) & 0x000F000Fu);
        const uint32_t h13 = opaque((w[i] >> 8) & 0x00F000F0u);
#pragma unroll
        for (int t = 0; t < NTK; ++t) {
            const float4* x4 = xv[t];
            lo_s[t] = __builtin_fmaf(half_of<0>(l02), x4[i].x, lo_s[t]);
            lo_s[t] = __builtin_fmaf(half_of<1>(l02), x4[i].z, lo_s[t]);
            lo_s[t] = __builtin_fmaf(half_of<0>(l13), x4[i].y, lo_s[t]);
            lo_s[t] = __builtin_fmaf(half_of<1>(l13), x4[i].w, lo_s[t]);
            hi_s[t] = __builtin_fmaf(half_of<0>(h02), x4[4 + i].x, hi_s[t]);
            hi_s[t] = __builtin_fmaf(half_of<1>(h02), x4[4 + i].z, hi_s[t]);
            hi_s[t] = __builtin_fmaf(half_of<0>(h13), x4[4 + i].y, hi_s[t]);
            hi_s[t] = __builtin_fmaf(half_of<1>(h13), x4[4 + i].w, hi_s[t]);
        }
    }
#pragma unroll
    for (int t = 0; t < NTK; ++t) out[t] = __builtin_fmaf(hi_s[t], 0.0625f, lo_s[t]);  // high nibbles read as 16q
}

// Per-lane constants of the Q4_K-style scale fields: sc_j sits at record bit
// ts = 6j and m_j at bit 32 + tm, tm = 16 + 6j. A field inside one word is cut
// out of that word rotated (v_alignbit_b32 of the word with itself), a field
// across two words out of the pair, so each field takes one select of the low
// source word, fixed per lane.
struct SubBlock {
    uint32_t ts, tm;
    bool sl, ml;
    __device__ explicit SubBlock(int j)
        : ts(6u * (uint32_t)j), tm(16u + 6u * (uint32_t)j), sl(6 * j < 32), ml(16 + 6 * j < 32) {}
};

// acc[t] += (Q4_0 contribution of the lane for token t) * 2^-24:
// d * (sum q*x_t - 8 * sum x_t).
template <int NTK>
__device__ __forceinline__ void dot24(const Traits<LW_Q4_0>::Packet& p, const float4* const* xv,
                                      const float* sx24, const SubBlock&, float* acc) {
    float qx[NTK];
    nibble_dot24<NTK>(p.c, xv, qx);
    const float d = half_bits_to_float(p.d);
#pragma unroll
    for (int t = 0; t < NTK; ++t) acc[t] = __builtin_fmaf(d, __builtin_fmaf(-8.0f, sx24[t], qx[t]), acc[t]);
}

// acc[t] += (q1_0 contribution of the lane for token t) * 2^-24:
// d * (2 * sum b*x_t - sum x_t); the masks of the 16 bit pairs serve every
// token, x_t pre-scaled by q1_prescale (so each masked bit times its x is
// b * x * 2^-24, as in bit_dot_pre).
template <int NTK>
__device__ __forceinline__ void dot24(const Traits<LW_Q1_0>::Packet& p, const float4* const* xv,
                                      const float* sx24, const SubBlock&, float* acc) {
    float lo_s[NTK], hi_s[NTK];
#pragma unroll
    for (int t = 0; t < NTK; ++t) lo_s[t] = hi_s[t] = 0.f;
    const uint32_t w4 = p.b >> 4;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const uint32_t m = q1_mask(p.b, w4, i);
        const int c = i & 3;
#pragma unroll
        for (int t = 0; t < NTK; ++t) {
            const float4& xl = xv[t][i >> 2];
            const float4& xh = xv[t][4 + (i >> 2)];
            lo_s[t] = __builtin_fmaf(half_of<0>(m), c == 0 ? xl.x : c == 1 ? xl.y : c == 2 ? xl.z : xl.w, lo_s[t]);
            hi_s[t] = __builtin_fmaf(half_of<1>(m), c == 0 ? xh.x : c == 1 ? xh.y : c == 2 ? xh.z : xh.w, hi_s[t]);
        }
    }
    const float d = half_bits_to_float(p.d);
#pragma unroll
    for (int t = 0; t < NTK; ++t) acc[t] = __builtin_fmaf(d, __builtin_fmaf(2.0f, lo_s[t] + hi_s[t], -sx24[t]), acc[t]);
}

// acc[t] += (Q4_1 contribution of the lane for token t) * 2^-24:
// d * sum q*x_t + m * sum x_t.
template <int NTK>
__device__ __forceinline__ void dot24(const Traits<LW_Q4_1>::Packet& p, const float4* const* xv,
                                      const float* sx24, const SubBlock&, float* acc) {
    float qx[NTK];
    nibble_dot24<NTK>(p.c, xv, qx);
    const float d = half_bits_to_float(p.dm & 0xFFFFu), m = half_bits_to_float(p.dm >> 16);
#pragma unroll
    for (int t = 0; t < NTK; ++t) acc[t] = __builtin_fmaf(m, sx24[t], __builtin_fmaf(d, qx[t], acc[t]));
}

// acc[t] += (Q4_K-style contribution for token t) * 2^-24:
// d*sc_j * sum q*x_t - dmin*m_j * sum x_t.
template <int NTK>
__device__ __forceinline__ void dot24(const Traits<LW_Q4_K>::Packet& p, const float4* const* xv,
                                      const float* sx24, const SubBlock& sb, float* acc) {
    const uint32_t sc_w = __builtin_amdgcn_alignbit(p.r1, sb.sl ? p.r0 : p.r1, sb.ts & 31u);
    const uint32_t m_w = __builtin_amdgcn_alignbit(p.r2, sb.ml ? p.r1 : p.r2, sb.tm & 31u);
    // d * sc and dmin * m, each one v_fma_mix with the binary16 operand (a +0
    // addend, which the compiler keeps; only an exact -0 product turns +0)
    const float ds = __builtin_fmaf(half_of<0>(p.dd), (float)(sc_w & 63u), 0.0f);
    const float dm = __builtin_fmaf(half_of<1>(p.dd), (float)(m_w & 63u), 0.0f);
    float qx[NTK];
    nibble_dot24<NTK>(p.c, xv, qx);
#pragma unroll
    for (int t = 0; t < NTK; ++t) acc[t] = __builtin_fmaf(-dm, sx24[t], __builtin_fmaf(ds, qx[t], acc[t]));
}

// Sums over the 64 lanes of NR accumulators at once: v_permlane32_swap and
// v_permlane16_swap fold the halves of different accumulators into one
// register, then DPP adds finish inside 16-lane (or 8-lane) rows. NR is
// padded with zeros to 1, 2, 4 or 8. The total of accumulator i lands in lane
// lane_of<NR>(i) of the returned register: NR = 1: lane 63; NR = 2: lanes 31,
// 63; NR = 4: lanes 15, 47, 31, 63; NR = 8: lanes 7, 39, 23, 55 (i < 4) and
// 15, 47, 31, 63 (i >= 4).
template <int NR>
constexpr int padded_rows() {
    return NR <= 1 ? 1 : NR <= 2 ? 2 : NR <= 4 ? 4 : 8;
}

template <int NR>
__device__ __forceinline__ int lane_of(int i) {
    constexpr int P = padded_rows<NR>();
    const int r16 = 2 * (i & 1) + ((i >> 1) & 1);  // 16-lane row of accumulator i (P = 4, 8)
    if constexpr (P == 1) return 63;
    else if constexpr (P == 2) return 32 * i + 31;
    else if constexpr (P == 4) return 16 * r16 + 15;
    else return 16 * r16 + (i < 4 ? 7 : 15);
}

__device__ __forceinline__ float fswap32(float a, float b, float& hi) {
    const auto s = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b),
                                                    false, false);
    hi = __builtin_bit_cast(float, (uint32_t)s[1]);
    return __builtin_bit_cast(float, (uint32_t)s[0]);
}

__device__ __forceinline__ float fswap16(float a, float b, float& odd) {
    const auto s = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b),
                                                    false, false);
    odd = __builtin_bit_cast(float, (uint32_t)s[1]);
    return __builtin_bit_cast(float, (uint32_t)s[0]);
}

// Four accumulators -> one register whose 16-lane rows hold accumulators 0,
// 2, 1, 3, each folded to 16 lanes.
__device__ __forceinline__ float fold4(float a0, float a1, float a2, float a3) {
    float h01, h23, o;
    const float l01 = fswap32(a0, a1, h01);
    const float l23 = fswap32(a2, a3, h23);
    const float e = fswap16(l01 + h01, l23 + h23, o);
    return e + o;
}

template <int NR>
__device__ __forceinline__ float rows_sum(const float* acc) {
    constexpr int P = padded_rows<NR>();
    float a[P];
#pragma unroll
    for (int i = 0; i < P; ++i) a[i] = i < NR ? acc[i] : 0.f;
    if constexpr (P == 1) {
        return wave_sum_to_lane63(a[0]);
    } else if constexpr (P == 2) {
        float h;
        const float l = fswap32(a[0], a[1], h);
        float v = l + h;  // lanes 0-31: accumulator 0 folded to 32 lanes; 32-63: accumulator 1
        v += dpp_move<0x111>(v);
        v += dpp_move<0x112>(v);
        v += dpp_move<0x114>(v);
        v += dpp_move<0x118>(v);
        v += dpp_move<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
        return v;
    } else if constexpr (P == 4) {
        float v = fold4(a[0], a[1], a[2], a[3]);
        v += dpp_move<0x111>(v);
        v += dpp_move<0x112>(v);
        v += dpp_move<0x114>(v);
        v += dpp_move<0x118>(v);
        return v;
    } else {
        const float r0 = fold4(a[0], a[1], a[2], a[3]);
        const float r1 = fold4(a[4], a[5], a[6], a[7]);
        // lanes 0-7 of each 16-lane row fold r0's row, lanes 8-15 fold r1's
        // (row_ror:8 brings the other half of the row)
        const bool upper = (__lane_id() & 8) != 0;
        const float t = upper ? r1 : r0, u = upper ? r0 : r1;
        float v = t + dpp_move<0x128>(u);
        v += dpp_move<0x111>(v);
        v += dpp_move<0x112>(v);
        v += dpp_move<0x114>(v);
        return v;
    }
}

template <int FMT, int NT, int R, int NW>
__global__ void __launch_bounds__(NW * kWave)
    gemv_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y,
                int64_t M, int64_t K, int KT, int64_t off1, int64_t off2, int64_t off3) {
    using T = Traits<FMT>;
    constexpr int EPL = T::EPL;
    constexpr int J4 = EPL / 4;  // float4s of x per lane per chunk
    constexpr int E = kWave * EPL;
    extern __shared__ float4 smem[];

    // token block blockIdx.y: tokens [NT * blockIdx.y, NT * blockIdx.y + NT)
    x += (int64_t)blockIdx.y * NT * K;
    y += (int64_t)blockIdx.y * NT * M;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t row_base = ((int64_t)blockIdx.x * NW + wave) * R;
    if (KT <= 0) return;               // never launched so; keeps the tile loop finite
    const int nch = (KT + E - 1) / E;  // chunks in a full tile
    const int tok4 = nch * E / 4;      // float4s per token in the LDS tile
    float4* xs = smem;
    float* sxs = reinterpret_cast<float*>(smem + NT * tok4);  // [NT][nch * 64] group sums

    int64_t rows[R];
#pragma unroll
    for (int r = 0; r < R; ++r) rows[r] = (row_base + r < M) ? row_base + r : M - 1;

    float acc[R][NT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[r][t] = 0.f;

    for (int64_t k0 = 0; k0 < K; k0 += KT) {
        const int kt = (int)((K - k0) < KT ? (K - k0) : KT);
        if (k0) __syncthreads();  // every wave is done with the previous tile
        // Stage x[:, k0 : k0+kt] (coalesced global reads, lane-interleaved LDS order).
        const int n4 = kt / 4;
        for (int idx = threadIdx.x; idx < NT * n4; idx += NW * kWave) {
            const int t = idx / n4, q = idx - t * n4;
            const int k = 4 * q;
            const int c = k / E, w = k - c * E, l = w / EPL, j4 = (w - l * EPL) / 4;
            xs[t * tok4 + (c * J4 + j4) * kWave + l] =
                *reinterpret_cast<const float4*>(x + (int64_t)t * K + k0 + k);
        }
        __syncthreads();
        if constexpr (T::kGroupSums) {
            const int ng = kt / 32;
            for (int idx = threadIdx.x; idx < NT * ng; idx += NW * kWave) {
                const int t = idx / ng, g = idx - t * ng;
                const int c = g / kWave, l = g - c * kWave;
                float s = 0.f;
#pragma unroll
                for (int j4 = 0; j4 < 8; ++j4) {
                    const float4 v = xs[t * tok4 + (c * 8 + j4) * kWave + l];
                    s += (v.x + v.y) + (v.z + v.w);
                }
                sxs[t * nch * kWave + g] = s;
            }
            __syncthreads();
        }

        const int nc = (kt + E - 1) / E;
        for (int c = 0; c < nc; ++c) {
            const int kl = c * E + lane * EPL;  // first element of the lane, within the tile
            if (kl < kt) {
                const int64_t kk = k0 + kl;
                typename T::Packet pk[R];
#pragma unroll
                for (int r = 0; r < R; ++r) pk[r] = T::load(W, rows[r] * K + kk, off1, off2, off3);
                const int j = (int)((kk >> 5) & 7);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    float4 xv[J4];
#pragma unroll
                    for (int j4 = 0; j4 < J4; ++j4) xv[j4] = xs[t * tok4 + (c * J4 + j4) * kWave + lane];
                    const float sx = T::kGroupSums ? sxs[t * nch * kWave + c * kWave + lane] : 0.f;
#pragma unroll
                    for (int r = 0; r < R; ++r) acc[r][t] += T::dot(pk[r], xv, sx, j);
                }
            }
        }
    }

#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float v = wave_sum_to_lane63(acc[r][t]);
            if (lane == kWave - 1 && row_base + r < M) y[(int64_t)t * M + row_base + r] = v;
        }
}

// Single-token kernel. The workgroup is persistent: it stages x once and then
// walks row batches (R rows) with a stride of the whole grid. A batch is one
// chunk-sized step per chunk of the row; the wave's steps over all its batches
// form one sequence, and the packets of the next D steps of that sequence are
// always in flight (a ring of D packet sets, refilled as each is consumed), so
// a wave keeps D * R * 1 KiB of weights outstanding across row boundaries. To
// keep the start short, every thread first issues its x loads, then the loads
// of its first D steps, and only then waits for x (vector-memory results
// return in issue order), so the x tile and its group sums are in LDS after
// one barrier while the weights are still on their way.
template <int FMT, int R, int D, int NW, int NS>
__global__ void __launch_bounds__(NW * kWave)
    gemv1_kernel(const RowSegs<NS> sg, const float* __restrict__ x, int64_t M, int64_t K) {
    using T = Traits<FMT>;
    using Packet = typename T::Packet;
    constexpr int EPL = T::EPL;
    constexpr int J4 = EPL / 4;
    constexpr int E = kWave * EPL;
    extern __shared__ float4 smem[];

    const int lane = threadIdx.x & (kWave - 1);
    // wave-uniform (the compiler cannot tell on its own): all row and plane
    // offsets derived from it live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int nc = (int)((K + E - 1) / E);  // chunks per row = steps per batch
    float4* xs = smem;                                          // nc * E floats, lane-interleaved
    float* sxs = reinterpret_cast<float*>(smem + nc * (E / 4));  // nc * 64 group sums (4-bit formats)
    float* sxs16 = sxs + nc * kWave;                              // Q2_K: sums of each group's first 16
    const int64_t nbatch = (M + R - 1) / R;
    const int64_t bstride = (int64_t)gridDim.x * NW;
    const int64_t b0 = (int64_t)blockIdx.x * NW + wave;
    const int nbw = b0 < nbatch ? (int)((nbatch - b0 + bstride - 1) / bstride) : 0;  // batches of this wave

    // (1) x loads first: thread t owns lane-slices t, t + blockDim, ... (EPL floats each).
    const int nsl = (int)(K / EPL);
    const int t0 = threadIdx.x;
    float4 xr[J4];
    if (t0 < nsl) {
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) xr[j4] = *reinterpret_cast<const float4*>(x + (int64_t)EPL * t0 + 4 * j4);
    }

    // (2) the first D steps. Every issue loads: a step past the wave's end
    // reads chunk 0 of row 0 and its packet is never used; in a chunk that
    // runs past K the lanes beyond it reload the last valid lane's bytes. So
    // the loads are unconditional and the compiler can count them, keeping
    // the next steps in flight while one is consumed.
    const uint32_t K32 = (uint32_t)K;
    const int total = nbw * nc;  // steps of this wave
    const uint32_t ulane = (uint32_t)lane;
    Packet ring[D][R];
    int ik = 0, ic = 0;  // next step to issue: batch ik of the wave, chunk ic
    auto issue = [&](Packet* pk) {
        const bool live = ik < nbw;
        const int64_t bb = b0 + (int64_t)ik * bstride;
        const uint32_t cc = live ? (uint32_t)ic : 0u;
        const uint32_t lmax = (K32 - cc * E) / EPL - 1u;  // last lane inside K
        const uint32_t la = ulane < lmax ? ulane : lmax;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t rr = bb * R + r;
            const int64_t row = live ? (rr < M ? rr : M - 1) : 0;
            const int si = seg_of(sg, row);
            const uint8_t* Ws = sg.W[si];
            pk[r] = T::load_at(Ws, Ws + sg.off1[si], Ws + sg.off2[si],
                               T::base((uint32_t)(row - sg.start[si]), K32, cc), la, Ws + sg.off3[si]);
        }
        if (++ic == nc) {
            ic = 0;
            ++ik;
        }
    };
#pragma unroll
    for (int d = 0; d < D; ++d) issue(ring[d]);

    // (3) x into LDS (and the group sums), one barrier
    auto put_slice = [&](int t, const float4* v) {
        const int c = t / kWave, l = t - c * kWave;
        float sum = 0.f;
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) sum += (v[j4].x + v[j4].y) + (v[j4].z + v[j4].w);
        if constexpr (FMT == LW_Q1_0 || FMT == LW_Q2_K) {
            // the 1- and 2-bit dots read x pre-scaled (the sums stay those of x)
            float4 u[J4];
#pragma unroll
            for (int j4 = 0; j4 < J4; ++j4) u[j4] = v[j4];
            if constexpr (FMT == LW_Q1_0) {
                q1_prescale(u);
            } else {
                sxs16[t] = sum16(v);
                q2_prescale(u);
            }
#pragma unroll
            for (int j4 = 0; j4 < J4; ++j4) xs[(c * J4 + j4) * kWave + l] = u[j4];
        } else {
#pragma unroll
            for (int j4 = 0; j4 < J4; ++j4) xs[(c * J4 + j4) * kWave + l] = v[j4];
        }
        if (T::kGroupSums) sxs[t] = sum;
    };
    if (t0 < nsl) put_slice(t0, xr);
    for (int t = t0 + NW * kWave; t < nsl; t += NW * kWave) {
        float4 v[J4];
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) v[j4] = *reinterpret_cast<const float4*>(x + (int64_t)EPL * t + 4 * j4);
        put_slice(t, v);
    }
    __syncthreads();

    // (4) consume the steps in order, refilling each ring slot D steps ahead.
    // Steady rounds (every refill is a real step) are straight-line code with
    // unconditional loads; only the last two rounds test what to refill.
    const int j = lane & 7;
    int k = 0, c = 0;  // step being consumed: batch k of the wave, chunk c
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
    auto consume = [&](const Packet* pk, bool live) {
        const bool ok = live && (uint32_t)(c * E + lane * EPL) < K32;
        float4 xv[J4];
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) xv[j4] = xs[(c * J4 + j4) * kWave + lane];
        const float sx = T::kGroupSums ? sxs[c * kWave + lane] : 0.f;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float v;
            if constexpr (FMT == LW_Q1_0)
                v = T::dot_pre(pk[r], xv, sx);
            else if constexpr (FMT == LW_Q2_K)
                v = T::dot_pre(pk[r], xv, sx, sxs16[c * kWave + lane]);
            else
                v = T::dot(pk[r], xv, sx, j);
            acc[r] += ok ? v : 0.f;
        }
    };
    auto finish_step = [&](bool live) {
        if (live && c == nc - 1) {
            const int64_t bb = b0 + (int64_t)k * bstride;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const float v = wave_sum_to_lane63(acc[r]);
                const int64_t row = bb * R + r;
                if (lane == kWave - 1 && row < M) {
                    const int si = seg_of(sg, row);
                    sg.y[si][row - sg.start[si]] = v;
                }
                acc[r] = 0.f;
            }
        }
        if (++c == nc) {
            c = 0;
            ++k;
        }
    };
    int s0 = 0;
    for (; s0 + 2 * D <= total; s0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            consume(ring[d], true);
            issue(ring[d]);
            finish_step(true);
        }
    }
#pragma unroll
    for (int d = 0; d < D; ++d) {
        const bool live = s0 + d < total;
        consume(ring[d], live);
        if (s0 + d + D < total) issue(ring[d]);
        finish_step(live);
    }
#pragma unroll
    for (int d = 0; d < D; ++d) {
        const bool live = s0 + D + d < total;
        if (live) {
            consume(ring[d], true);
            finish_step(true);
        }
    }
}

// Group sum over aligned 8-lane groups: lane 8m+7 ends with the sum of
// lanes 8m..8m+7 (row_shr 1, 2, 4 inside each 16-lane row).
__device__ __forceinline__ float sum8_to_last(float v) {
    v += dpp_move<0x111>(v);
    v += dpp_move<0x112>(v);
    v += dpp_move<0x114>(v);
    return v;
}

// Kernel for one to a few tokens over the 4-bit formats with the activation
// held in registers. K is a whole number NC of chunks (2048 elements); a
// workgroup is G row groups x WPR waves, and wave w of a row group owns chunks
// [w*CPW, (w+1)*CPW) of every row of that group (NC = CPW*WPR), so lane l
// keeps x_t[c*2048 + 32l : +32] and its group sum, for each of the NTK tokens
// and those CPW chunks, in VGPRs for the whole kernel and never reads x
// again; the nibble masks of a packet serve all tokens. The rows of row group
// rg = blockIdx.x*G + g are rg, rg + gridDim.x*G, ...; each wave keeps the
// packets of its next DR rows in flight (a ring refilled as each row is
// consumed) and sums its DR x NTK (row, token) accumulators over the 64 lanes
// at once. With WPR == 1 the wave stores the totals; with WPR > 1 each wave's
// per-row partials go to LDS and the WPR partials of an output are added in
// wave order after one barrier at the end. x is staged once: coalesced
// 16-byte loads (issued before the first rows' packets), group sums by DPP
// over the 8 lanes that hold one group, an LDS tile in which float4 j4 of
// lane l of chunk c of token t sits at row (t*NC + c)*8 + j4, column l ^ j4
// (the 8 lanes that stage one group write 8 different bank groups, and the 64
// lanes reading one row read 64 different float4s), one barrier, then one
// read per lane.
template <int FMT, int NTK, int CPW, int WPR, int G, int DR, int NS>
__global__ void __launch_bounds__(G * WPR * kWave)
    gemv1r_kernel(const RowSegs<NS> sg, const float* __restrict__ x, int M, int nr_max) {
    using T = Traits<FMT>;
    using Packet = typename T::Packet;
    static_assert(T::EPL == 32 && T::kGroupSums, "4-bit formats only");
    constexpr int J4 = 8;                      // float4s of x per lane per chunk
    constexpr int E = kWave * 32;              // elements per chunk
    constexpr int NC = CPW * WPR;              // chunks per row
    constexpr uint32_t K = (uint32_t)NC * E;
    constexpr int NTH = G * WPR * kWave;       // threads per workgroup
    constexpr int NQ = NTK * (int)(K / 4);     // float4s of x (all tokens)
    constexpr int XPT = (NQ + NTH - 1) / NTH;  // x float4s per thread
    constexpr int NR = DR * NTK;               // (row, token) sums per round
    static_assert(NTH % kWave == 0 && NQ % 8 == 0, "group sums need whole 8-lane groups");
    static_assert(NR <= 8, "at most 8 lane sums per round");
    extern __shared__ float4 smem[];
    float4* xs = smem;                                 // NQ float4s
    float* sxs = reinterpret_cast<float*>(smem + NQ);  // NTK * NC * 64 group sums
    float* red = sxs + NTK * NC * kWave;               // [G][nr_max][NTK][WPR] partials

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int g = wv / WPR, w = wv - g * WPR;
    const int rg = blockIdx.x * G + g;
    const int rgs = gridDim.x * G;
    const int nr = rg < M ? (M - 1 - rg) / rgs + 1 : 0;  // rows of this row group

    // (1) x loads (clamped index: every load is issued)
    float4 xv[XPT];
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
        const int q = tid + i * NTH;
        xv[i] = *reinterpret_cast<const float4*>(x + 4 * (q < NQ ? q : NQ - 1));
    }

    // (2) packets of the first DR rows. A row index past the group's end loads
    // row 0 and its packets are never used.
    const uint32_t ulane = (uint32_t)lane;
    Packet ring[DR][CPW];
    int ik = 0;  // next row (of the group) to issue
    auto issue = [&](Packet* pk) __attribute__((always_inline)) {
        const int row = ik < nr ? rg + ik * rgs : 0;
        const int si = seg_of(sg, row);
        const uint8_t* Ws = sg.W[si];
        const uint8_t* P1 = Ws + sg.off1[si];
        const uint8_t* P2 = Ws + sg.off2[si];
        const uint32_t lr = (uint32_t)(row - (int)sg.start[si]);
#pragma unroll
        for (int cc = 0; cc < CPW; ++cc)
            pk[cc] = T::load_at(Ws, P1, P2, T::base(lr, K, (uint32_t)(w * CPW + cc)), ulane);
        ++ik;
    };
#pragma unroll
    for (int d = 0; d < DR; ++d) issue(ring[d]);

    // (3) x into LDS with its group sums, one barrier, then this lane's slices.
    // Float4 q of x is token q / (K/4), chunk (q mod K/4) / 512 of it.
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
        const int q = tid + i * NTH;
        const int tc = q / (E / 4), rem = q - tc * (E / 4), l = rem / J4, j4 = rem - l * J4;
        const float s = sum8_to_last((xv[i].x + xv[i].y) + (xv[i].z + xv[i].w));
        if (q < NQ) {
            xs[(tc * J4 + j4) * kWave + (l ^ j4)] = xv[i];
            if ((tid & 7) == 7) sxs[q / J4] = s;
        }
    }
    __syncthreads();
    float4 xr[NTK][CPW][J4];
    float sx24[NTK][CPW];
#pragma unroll
    for (int t = 0; t < NTK; ++t)
#pragma unroll
        for (int cc = 0; cc < CPW; ++cc) {
            const int tc = t * NC + w * CPW + cc;
#pragma unroll
            for (int j4 = 0; j4 < J4; ++j4) xr[t][cc][j4] = xs[(tc * J4 + j4) * kWave + (lane ^ j4)];
            if constexpr (FMT == LW_Q1_0) q1_prescale(xr[t][cc]);  // the 1-bit dot's form
            sx24[t][cc] = sxs[tc * kWave + lane] * 5.9604644775390625e-8f;  // 2^-24
        }

    // (4) consume rows in order, DR at a time, refilling each ring slot DR
    // rows ahead. Steady rounds refill only real rows, so their loads are
    // unconditional; the last two rounds test what to consume and refill.
    const SubBlock sb(lane & 7);  // the lane's sub-block within a super-block
    int my_i = -1;  // the (row, token) sum this lane receives: i = d * NTK + t
#pragma unroll
    for (int i = 0; i < NR; ++i)
        if (lane == lane_of<NR>(i)) my_i = i;
    const int my_d = my_i / NTK, my_t = my_i - my_d * NTK;
    auto round = [&](int s0, bool steady) __attribute__((always_inline)) {
        float acc[NR];
#pragma unroll
        for (int d = 0; d < DR; ++d) {
#pragma unroll
            for (int t = 0; t < NTK; ++t) acc[d * NTK + t] = 0.f;
            if (steady || s0 + d < nr) {
#pragma unroll
                for (int cc = 0; cc < CPW; ++cc) {
                    const float4* xp[NTK];
                    float s24[NTK];
#pragma unroll
                    for (int t = 0; t < NTK; ++t) {
                        xp[t] = xr[t][cc];
                        s24[t] = sx24[t][cc];
                    }
                    dot24<NTK>(ring[d][cc], xp, s24, sb, acc + d * NTK);
                }
            }
            if (steady || s0 + d + DR < nr) issue(ring[d]);
        }
        const float v = rows_sum<NR>(acc) * 16777216.0f;  // 2^24
        const int kk = s0 + my_d;
        if (my_i >= 0 && kk < nr) {
            if constexpr (WPR == 1) {
                const int row = rg + kk * rgs;
                const int si = seg_of(sg, row);
                sg.y[si][(int64_t)my_t * sg.M[si] + (row - sg.start[si])] = v;
            } else
                red[((g * nr_max + kk) * NTK + my_t) * WPR + w] = v;
        }
    };
    int s0 = 0;
    for (; s0 + 2 * DR <= nr; s0 += DR) round(s0, true);
    round(s0, false);
    round(s0 + DR, false);

    if constexpr (WPR > 1) {
        __syncthreads();
        for (int idx = tid; idx < G * nr_max * NTK; idx += NTH) {
            const int t = idx % NTK, gi = idx / NTK;
            const int gg = gi / nr_max, ii = gi - gg * nr_max;
            const int64_t row = (int64_t)blockIdx.x * G + gg + (int64_t)ii * rgs;
            if (row < M) {
                float s = 0.f;
#pragma unroll
                for (int ww = 0; ww < WPR; ++ww) s += red[idx * WPR + ww];
                const int si = seg_of(sg, row);
                sg.y[si][(int64_t)t * sg.M[si] + (row - sg.start[si])] = s;
            }
        }
    }
}

struct Config {
    int R, NW;
};

// ntb token blocks of NT tokens each (x and y advance by NT rows per block),
// one launch: grid.y is the token block.
template <int FMT, int NT>
hipError_t launch_nt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                     const Planes& p, hipStream_t stream, int64_t ntb = 1) {
    constexpr int E = kWave * Traits<FMT>::EPL;
    constexpr int R = NT == 1 ? 4 : (NT <= 4 ? 2 : 1);
    constexpr int NW = 4;
    // x tile: the whole K if it fits the LDS budget, else the largest whole
    // number of chunks that does (each chunk: NT x E floats of x, plus NT x 64
    // group sums for the 4-bit formats).
    const int64_t chunk_bytes = (int64_t)NT * (E * 4 + (Traits<FMT>::kGroupSums ? kWave * 4 : 0));
    int64_t nch = (K + E - 1) / E;
    if (nch * chunk_bytes > kLdsBytes) nch = kLdsBytes / chunk_bytes;
    if (nch < 1) return hipErrorInvalidConfiguration;  // callers split tokens first (see fits_one_chunk)
    const int64_t KT = nch * E;
    const size_t lds = (size_t)(nch * chunk_bytes);
    const int64_t blocks = (M + (int64_t)NW * R - 1) / ((int64_t)NW * R);
    if (query_only(kernel_name<Name_gemv_kernel, FMT, NT, R, NW>())) return hipSuccess;
    hipLaunchKernelGGL((gemv_kernel<FMT, NT, R, NW>), dim3((unsigned)blocks, (unsigned)ntb), dim3(NW * kWave), lds,
                       stream, W, x, y, M, K, (int)KT, p.off1, p.off2, p.off3);
    return hipGetLastError();
}

// Whether one chunk of x for NT tokens (plus its group sums) fits the LDS budget.
template <int FMT, int NT>
constexpr bool fits_one_chunk() {
    return (int64_t)NT * (kWave * Traits<FMT>::EPL * 4 + (Traits<FMT>::kGroupSums ? kWave * 4 : 0)) <=
           kLdsBytes;
}

// Compute units of the current device, looked up once per device.
int cu_count() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v <= 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// Rows of one matrix as a one-segment row space.
inline RowSegs<1> one_seg(const uint8_t* W, float* y, int64_t M, const Planes& p) {
    RowSegs<1> sg;
    sg.W[0] = W;
    sg.y[0] = y;
    sg.off1[0] = p.off1;
    sg.off2[0] = p.off2;
    sg.off3[0] = p.off3;
    sg.start[0] = 0;
    sg.M[0] = M;
    return sg;
}

// Single token: the persistent kernel when the whole x row fits the LDS
// budget and every segment's planes stay below 4 GiB (32-bit offsets), else
// hipErrorNotSupported (a single matrix then takes the K-tiled kernel).
template <int FMT, int R, int D, int NS>
hipError_t launch_single_segs(const RowSegs<NS>& sg, const float* x, int64_t M, int64_t K, int64_t max_total,
                              hipStream_t stream) {
    constexpr int NW = 8;
    constexpr int E = kWave * Traits<FMT>::EPL;
    const int64_t nc = (K + E - 1) / E;
    const int64_t lds = nc * E * 4 + (Traits<FMT>::kGroupSums ? nc * kWave * 4 : 0) +
                        (FMT == LW_Q2_K ? nc * kWave * 4 : 0);  // Q2_K: the first-16 sums
    if (lds > kLdsBytes || max_total >= ((int64_t)1 << 32) || M >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    const int64_t nbatch = (M + R - 1) / R;
    int64_t grid = (nbatch + NW - 1) / NW;
    const int64_t cap = 2 * (int64_t)cu_count();  // two 8-wave workgroups per CU
    if (grid > cap) grid = cap;
    if (query_only(kernel_name<Name_gemv1_kernel, FMT, R, D, NW, NS>())) return hipSuccess;
    hipLaunchKernelGGL((gemv1_kernel<FMT, R, D, NW, NS>), dim3((unsigned)grid), dim3(NW * kWave), (size_t)lds,
                       stream, sg, x, M, K);
    return hipGetLastError();
}

// Rows per wave step (R) and ring depth (D) of the LDS single-token kernel,
// from MI355X sweeps: one row and two steps for the 4-bit formats and Q8_0
// (eight steps for q1_0, whose steps are a quarter of the bytes);
// f16 keeps four steps in flight (two rows each for 3072..8191 rows at
// K <= 2048, e.g. the 1B q/k/v projection).
template <int FMT, int NS>
hipError_t launch_single_table(const RowSegs<NS>& sg, const float* x, int64_t M, int64_t K, int64_t max_total,
                               hipStream_t stream) {
    if constexpr (FMT == LW_F16) {
        if (K <= 2048 && M >= 3072 && M < 8192) return launch_single_segs<FMT, 2, 4, NS>(sg, x, M, K, max_total, stream);
        return launch_single_segs<FMT, 1, 4, NS>(sg, x, M, K, max_total, stream);
    } else if constexpr (FMT == LW_Q1_0) {
        // a step is 256 bytes of bits per wave: keep eight of them in flight
        // (four rows per step, sharing each x read, leave too few waves with
        // work on 2048-row matrices and measured slower)
        return launch_single_segs<FMT, 1, 8, NS>(sg, x, M, K, max_total, stream);
    } else {
        return launch_single_segs<FMT, 1, 2, NS>(sg, x, M, K, max_total, stream);
    }
}

template <int FMT>
hipError_t launch_single(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                         const Planes& p, hipStream_t stream) {
    const hipError_t err = launch_single_table<FMT, 1>(one_seg(W, y, M, p), x, M, K, p.total, stream);
    if (err == hipErrorNotSupported) return launch_nt<FMT, 1>(W, x, y, M, K, p, stream);
    return err;
}

// Register-resident-x kernel: G row groups x WPR waves per workgroup, at most
// CAP workgroups per compute unit. Returns hipErrorNotSupported when the shape
// does not fit it (the caller then uses another kernel).
template <int FMT, int NTK, int CPW, int WPR, int G, int DR, int CAP, int NS>
hipError_t launch_reg(const RowSegs<NS>& sg, const float* x, int64_t M, int64_t max_total, hipStream_t stream) {
    constexpr int64_t NC = CPW * WPR;
    constexpr int64_t K = NC * kWave * 32;
    if (max_total >= ((int64_t)1 << 32) || M >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    int64_t grid = (M + G - 1) / G;
    const int64_t cap = CAP * (int64_t)cu_count();
    if (grid > cap) grid = cap;
    const int64_t nr_max = (M + grid * G - 1) / (grid * G);
    const int64_t lds = NTK * (K * 4 + NC * kWave * 4) + (WPR > 1 ? G * nr_max * NTK * WPR * 4 : 0);
    if (lds > kRegLdsBytes) return hipErrorNotSupported;
    if (query_only(kernel_name<Name_gemv1r_kernel, FMT, NTK, CPW, WPR, G, DR, NS>())) return hipSuccess;
    hipLaunchKernelGGL((gemv1r_kernel<FMT, NTK, CPW, WPR, G, DR, NS>), dim3((unsigned)grid),
                       dim3(G * WPR * kWave), (size_t)lds, stream, sg, x, (int)M, (int)nr_max);
    return hipGetLastError();
}

// Kernel selection for the register kernel over the 4-bit formats, by token
// count, the number of 2048-element chunks per row (K / 2048) and the row
// count. With one token the register kernel needs a few rows per wave to pay
// for staging x whole; below that (and for other K) the LDS kernel, which
// spreads single chunks over the waves, is faster.
// A register-kernel candidate of the selection table (select.hpp): the
// configuration it names when its chunk and token counts match the call,
// else hipErrorNotSupported.
template <int FMT, int NS>
hipError_t launch_reg_cand(int cand, const RowSegs<NS>& sg, const float* x, int64_t M, int64_t K, int64_t n_tok,
                           int64_t max_total, hipStream_t stream) {
    if (K % 2048) return hipErrorNotSupported;
    const int64_t nc = K / 2048;
    const bool t1 = n_tok == 1, t2 = n_tok == 2 && NS == 1;
    switch (cand) {
    case kCandReg1_1x1_G8_D2_C2:
        if (t1 && nc == 1) return launch_reg<FMT, 1, 1, 1, 8, 2, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x1_G4_D2_C4:
        if (t1 && nc == 1) return launch_reg<FMT, 1, 1, 1, 4, 2, 4, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x1_G8_D3_C2:
        if (t1 && nc == 1) return launch_reg<FMT, 1, 1, 1, 8, 3, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_2x1_G8_D2_C2:
        if (t1 && nc == 2) return launch_reg<FMT, 1, 2, 1, 8, 2, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x2_G4_D2_C2:
        if (t1 && nc == 2) return launch_reg<FMT, 1, 1, 2, 4, 2, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x2_G8_D2_C1:
        if (t1 && nc == 2) return launch_reg<FMT, 1, 1, 2, 8, 2, 1, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_2x1_G8_D3_C2:
        if (t1 && nc == 2) return launch_reg<FMT, 1, 2, 1, 8, 3, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_2x1_G4_D2_C4:
        if (t1 && nc == 2) return launch_reg<FMT, 1, 2, 1, 4, 2, 4, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x7_G2_D2_C1:
        if (t1 && nc == 7) return launch_reg<FMT, 1, 1, 7, 2, 2, 1, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x7_G1_D2_C2:
        if (t1 && nc == 7) return launch_reg<FMT, 1, 1, 7, 1, 2, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg1_1x7_G2_D3_C1:
        if (t1 && nc == 7) return launch_reg<FMT, 1, 1, 7, 2, 3, 1, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg2_1x1_G8_D2_C2:
        if (t2 && nc == 1) return launch_reg<FMT, 2, 1, 1, 8, 2, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg2_1x2_G4_D2_C2:
        if (t2 && nc == 2) return launch_reg<FMT, 2, 1, 2, 4, 2, 2, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg2_1x4_G2_D2_C1:
        if (t2 && nc == 4) return launch_reg<FMT, 2, 1, 4, 2, 2, 1, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg2_1x7_G2_D2_C1:
        if (t2 && nc == 7) return launch_reg<FMT, 2, 1, 7, 2, 2, 1, NS>(sg, x, M, max_total, stream);
        break;
    case kCandReg2_1x2_G8_D2_C1:
        if (t2 && nc == 2) return launch_reg<FMT, 2, 1, 2, 8, 2, 1, NS>(sg, x, M, max_total, stream);
        break;
    default:
        break;
    }
    return hipErrorNotSupported;
}

// Kernel selection for the register kernel over the 4-bit formats, by token
// count, the number of 2048-element chunks per row (K / 2048) and the row
// count: the swept table's candidate where it names one for the shape (the
// LDS candidate: hipErrorNotSupported, so the caller takes the LDS kernel),
// else the built-in rules. With one token the register kernel needs a few
// rows per wave to pay for staging x whole; below that (and for other K) the
// LDS kernel, which spreads single chunks over the waves, is faster.
template <int FMT, int NS>
hipError_t launch_reg_segs(const RowSegs<NS>& sg, const float* x, int64_t M, int64_t K, int64_t n_tok,
                           int64_t max_total, hipStream_t stream) {
    if (K % 2048) return hipErrorNotSupported;
    const int64_t nc = K / 2048;
    if constexpr (FMT == LW_Q1_0) {
        // one-chunk rows (K = 2048) only: a row is 256 bytes of bits per
        // wave, so each wave keeps four rows in flight
        if (nc == 1 && n_tok == 1) return launch_reg<FMT, 1, 1, 1, 8, 4, 2, NS>(sg, x, M, max_total, stream);
        if (nc == 1 && n_tok == 2 && NS == 1) return launch_reg<FMT, 2, 1, 1, 8, 4, 2, NS>(sg, x, M, max_total, stream);
        return hipErrorNotSupported;
    } else {
        const int cand = select_cand(FMT, M, K, n_tok);
        if (cand == kCandLds) return hipErrorNotSupported;
        if (is_reg_cand(cand)) {
            const hipError_t err = launch_reg_cand<FMT, NS>(cand, sg, x, M, K, n_tok, max_total, stream);
            if (err != hipErrorNotSupported) return err;
        }
        if (n_tok == 1) {
            if (nc == 1) return launch_reg<FMT, 1, 1, 1, 8, 2, 2, NS>(sg, x, M, max_total, stream);
            if (nc == 2 && M >= 10240) return launch_reg<FMT, 1, 2, 1, 8, 2, 2, NS>(sg, x, M, max_total, stream);
            if (nc == 7) return launch_reg<FMT, 1, 1, 7, 2, 2, 1, NS>(sg, x, M, max_total, stream);
        } else if (n_tok == 2 && NS == 1) {
            if (nc == 1) return launch_reg<FMT, 2, 1, 1, 8, 2, 2, NS>(sg, x, M, max_total, stream);
            if (nc == 2) return launch_reg<FMT, 2, 1, 2, 4, 2, 2, NS>(sg, x, M, max_total, stream);
            if (nc == 4) return launch_reg<FMT, 2, 1, 4, 2, 2, 1, NS>(sg, x, M, max_total, stream);
            if (nc == 7) return launch_reg<FMT, 2, 1, 7, 2, 2, 1, NS>(sg, x, M, max_total, stream);
        }
        return hipErrorNotSupported;
    }
}

template <int FMT>
hipError_t launch_reg_fmt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                          const Planes& p, hipStream_t stream) {
    return launch_reg_segs<FMT, 1>(one_seg(W, y, M, p), x, M, K, n_tok, p.total, stream);
}

// One launch over the rows of n matrices sharing x (one token): the register
// kernel's table for the total row count, else the LDS single-token kernel.
template <int FMT, int NS>
hipError_t launch_multi_ns(int n, const uint8_t* const* W, float* const* y, const int64_t* M, const float* x,
                           int64_t K, hipStream_t stream) {
    RowSegs<NS> sg;
    int64_t tot = 0, max_total = 0;
    for (int i = 0; i < NS; ++i) {
        const bool used = i < n;
        const Planes p = planes_of(FMT, used ? M[i] * K : 0);
        sg.W[i] = used ? W[i] : W[0];
        sg.y[i] = used ? y[i] : y[0];
        sg.off1[i] = p.off1;
        sg.off2[i] = p.off2;
        sg.off3[i] = p.off3;
        sg.start[i] = used ? tot : INT64_MAX;
        sg.M[i] = used ? M[i] : 0;
        if (used) {
            tot += M[i];
            if (p.total > max_total) max_total = p.total;
        }
    }
    if constexpr (FMT == LW_Q4_0 || FMT == LW_Q4_K || FMT == LW_Q4_1 || FMT == LW_Q1_0) {
        const hipError_t err = launch_reg_segs<FMT, NS>(sg, x, tot, K, 1, max_total, stream);
        if (err != hipErrorNotSupported) return err;
    }
    return launch_single_table<FMT, NS>(sg, x, tot, K, max_total, stream);
}

// Two matrices (a layer's gate and up) get a segment table of two, which
// keeps the per-row segment choice to one compare.
template <int FMT>
hipError_t launch_multi_fmt(int n, const uint8_t* const* W, float* const* y, const int64_t* M, const float* x,
                            int64_t K, hipStream_t stream) {
    if (n <= 2) return launch_multi_ns<FMT, 2>(n, W, y, M, x, K, stream);
    return launch_multi_ns<FMT, kMaxSegs>(n, W, y, M, x, K, stream);
}

template <int FMT>
hipError_t launch_fmt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                      int64_t n_tok, const Planes& p, hipStream_t stream) {
    if (n_tok == 1) return launch_single<FMT>(W, x, y, M, K, p, stream);
    if constexpr (!fits_one_chunk<FMT, 8>()) {
        // 8 tokens of a 4-bit chunk (64 KiB of x) plus group sums exceed the
        // budget: run them as two launches of 4 tokens.
        if (n_tok == 8) {
            hipError_t err = launch_nt<FMT, 4>(W, x, y, M, K, p, stream);
            if (err != hipSuccess) return err;
            return launch_nt<FMT, 4>(W, x + 4 * K, y + 4 * M, M, K, p, stream);
        }
    }
    switch (n_tok) {
    case 1: return launch_nt<FMT, 1>(W, x, y, M, K, p, stream);
    case 2: return launch_nt<FMT, 2>(W, x, y, M, K, p, stream);
    case 3: return launch_nt<FMT, 3>(W, x, y, M, K, p, stream);
    case 4: return launch_nt<FMT, 4>(W, x, y, M, K, p, stream);
    case 5: return launch_nt<FMT, 5>(W, x, y, M, K, p, stream);
    case 6: return launch_nt<FMT, 6>(W, x, y, M, K, p, stream);
    case 7: return launch_nt<FMT, 7>(W, x, y, M, K, p, stream);
    case 8:
        if constexpr (fits_one_chunk<FMT, 8>()) return launch_nt<FMT, 8>(W, x, y, M, K, p, stream);
        return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_gemv_multi(int fmt, int n, const uint8_t* const* W, float* const* y, const int64_t* M,
                             const float* x, int64_t K, hipStream_t stream) {
    switch (fmt) {
    case LW_F16: return launch_multi_fmt<LW_F16>(n, W, y, M, x, K, stream);
    case LW_Q8_0: return launch_multi_fmt<LW_Q8_0>(n, W, y, M, x, K, stream);
    case LW_Q4_0: return launch_multi_fmt<LW_Q4_0>(n, W, y, M, x, K, stream);
    case LW_Q4_K: return launch_multi_fmt<LW_Q4_K>(n, W, y, M, x, K, stream);
    case LW_Q4_1: return launch_multi_fmt<LW_Q4_1>(n, W, y, M, x, K, stream);
    case LW_Q1_0: return launch_multi_fmt<LW_Q1_0>(n, W, y, M, x, K, stream);
    case LW_Q5_0: return launch_multi_fmt<LW_Q5_0>(n, W, y, M, x, K, stream);
    case LW_Q5_1: return launch_multi_fmt<LW_Q5_1>(n, W, y, M, x, K, stream);
    case LW_Q5_K: return launch_multi_fmt<LW_Q5_K>(n, W, y, M, x, K, stream);
    case LW_Q6_K: return launch_multi_fmt<LW_Q6_K>(n, W, y, M, x, K, stream);
    case LW_Q2_K: return launch_multi_fmt<LW_Q2_K>(n, W, y, M, x, K, stream);
    case LW_MXFP4: return launch_multi_fmt<LW_MXFP4>(n, W, y, M, x, K, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemv_reg(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                           int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_reg_fmt<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_reg_fmt<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_reg_fmt<LW_Q4_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q1_0: return launch_reg_fmt<LW_Q1_0>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorNotSupported;
    }
}

// Any token count on the matrix-vector kernels: whole blocks of NT tokens
// (8, or 4 where 8 tokens of a chunk exceed the LDS budget) in one launch per
// 65535 blocks, the remaining tokens in one more.
template <int FMT>
hipError_t launch_blocks_fmt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                             const Planes& p, hipStream_t stream) {
    constexpr int NT = fits_one_chunk<FMT, 8>() ? 8 : 4;
    constexpr int64_t kMaxGridY = 65535;
    const int64_t nb = n_tok / NT;
    for (int64_t b0 = 0; b0 < nb; b0 += kMaxGridY) {
        const int64_t cnt = (nb - b0) < kMaxGridY ? (nb - b0) : kMaxGridY;
        const hipError_t err = launch_nt<FMT, NT>(W, x + b0 * NT * K, y + b0 * NT * M, M, K, p, stream, cnt);
        if (err != hipSuccess) return err;
    }
    const int64_t rem = n_tok - nb * NT;
    if (rem == 0) return hipSuccess;
    return launch_fmt<FMT>(W, x + nb * NT * K, y + nb * NT * M, M, K, rem, p, stream);
}

hipError_t launch_gemv_blocks(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                              int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_F16: return launch_blocks_fmt<LW_F16>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_blocks_fmt<LW_Q8_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_0: return launch_blocks_fmt<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_blocks_fmt<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_blocks_fmt<LW_Q4_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q1_0: return launch_blocks_fmt<LW_Q1_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_0: return launch_blocks_fmt<LW_Q5_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_1: return launch_blocks_fmt<LW_Q5_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_K: return launch_blocks_fmt<LW_Q5_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q6_K: return launch_blocks_fmt<LW_Q6_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q2_K: return launch_blocks_fmt<LW_Q2_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_MXFP4: return launch_blocks_fmt<LW_MXFP4>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemv(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                       int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_F16: return launch_fmt<LW_F16>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_fmt<LW_Q8_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_0: return launch_fmt<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_fmt<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_fmt<LW_Q4_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q1_0: return launch_fmt<LW_Q1_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_0: return launch_fmt<LW_Q5_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_1: return launch_fmt<LW_Q5_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_K: return launch_fmt<LW_Q5_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q6_K: return launch_fmt<LW_Q6_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q2_K: return launch_fmt<LW_Q2_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_MXFP4: return launch_fmt<LW_MXFP4>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
