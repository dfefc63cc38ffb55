// Prefill product on the matrix cores (many tokens; every quantized format).
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k]. With many tokens the product is
// a contraction over K with a token dimension, so it runs on the matrix cores
// (Sec. 3.2: matrix multiplication tiles through shared memory and uses the
// cooperative matrix instructions of the device; Sec. 3.3: quantized blocks
// are dequantized on the way in and each decoded tile is reused for every
// token of the workgroup): gemm32_kernel on v_mfma_f32_32x32x16_bf16 for the
// formats with at most 6-bit codes and MXFP4, gemm_kernel on
// v_mfma_f32_16x16x32_bf16 for Q8_0.
//
// Precision. The weight operand holds exact bfloat16 values derived from the
// integer codes only: the biased code 128 + q (bits 0x4300 | q, q < 64) for
// the formats with an offset, the code q for Q8_0, the e2m1 value for MXFP4,
// +-1 for q1_0.
// X is split into bf16 high and low parts (x = hi + lo to 2^-17 relative),
// two MFMAs per tile and K-step, float32 accumulation. A coefficient unit
// (a 32-element block, or a 16-element sub-block for Q6_K and Q2_K) applies
// its scale, min and bias to its float32 partial P:
//   Q4_0:   y += d * P - 136 * d * S             (128 + q = (q - 8) + 136)
//   Q5_0:   y += d * P - 144 * d * S             (128 + q = (q - 16) + 144)
//   Q4_1, Q5_1:  y += d * P + (m - 128*d) * S
//   Q4_K, Q5_K:  y += d*sc * P - (128*d*sc + dmin*m) * S
//   Q6_K:   y += d*sc * P - 160 * d*sc * S       (128 + q = (q - 32) + 160)
//   Q2_K:   y += d*sc * P - (128*d*sc + dmin*m) * S
//   Q8_0, q1_0:  y += d * P;   MXFP4:  y += 2^(E - 127) * P
// where S = sum over the unit of (hi + lo), the very values fed to the
// matrix core, so the bias cancels to float32 rounding. The error relative
// to sum_k |w * x| stays near 1e-5.
//
// Layout of one block in the 16 x 16 x 32 operands: lane slice s (lanes
// 16s..16s+15) holds 8 of the block's 32 elements (Q8_0: elements 8s..8s+7).
// The 32 x 32 x 16 layout is described at gemm32_kernel. The X operand in LDS
// uses the same order of k.
#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

// names of the kernel templates, for lw_kernel_name
struct Name_gemm_kernel {
    static constexpr const char* base = "gemm_kernel";
};
struct Name_gemm32_kernel {
    static constexpr const char* base = "gemm32_kernel";
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));


// x = hi + lo with hi = bf16(x) (round to nearest even) and lo = bf16(x - hi);
// returns the float sum of the 8 (hi + lo). Pairs are converted with one
// v_cvt_pk_bf16_f32 each; a bf16 widens to float by a shift or a mask.
__device__ __forceinline__ float split_bf16x8(const float* v, bf16x8* h, bf16x8* l) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 hw, lw;
    float sum = 0.f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t hb = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{v[2 * p], v[2 * p + 1]}), bf16x2));
        const float h0 = __builtin_bit_cast(float, hb << 16), h1 = __builtin_bit_cast(float, hb & 0xFFFF0000u);
        const uint32_t lb = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{v[2 * p] - h0, v[2 * p + 1] - h1}), bf16x2));
        const float l0 = __builtin_bit_cast(float, lb << 16), l1 = __builtin_bit_cast(float, lb & 0xFFFF0000u);
        sum += (h0 + l0) + (h1 + l1);
        hw[p] = hb;
        lw[p] = lb;
    }
    *h = __builtin_bit_cast(bf16x8, hw);
    *l = __builtin_bit_cast(bf16x8, lw);
    return sum;
}

template <int FMT>
struct MF;

// 4-bit formats: code word of (row, block, slice), biased bf16 codes.
template <int FMT>
struct MF4 {
    static constexpr bool kSums = true;
    static constexpr int kRaw = FMT == LW_Q4_1 ? 8 : 4;  // raw scale words of 8 blocks
    __device__ static uint32_t code_word(const uint8_t* W, uint64_t row, uint32_t K, int blk, int s) {
        return *reinterpret_cast<const uint32_t*>(W + row * (K / 2u) + 16u * (uint32_t)blk + 4u * s);
    }
    // 128 + q as bf16: bits 0x4300 | q. Pair p of the operand = nibbles (p, p+4)
    // of the word would need shifts; the order below keeps element order
    // (lo nibbles of bytes 0..3, then hi nibbles), matching x_first().
    __device__ static bf16x8 decode(uint32_t w) {
        const uint32_t lo = opaque(w & 0x0F0F0F0Fu);         // bytes: q of elements 4s..4s+3
        const uint32_t hi = opaque((w >> 4) & 0x0F0F0F0Fu);  // bytes: q of elements 16+4s..
        // v_perm_b32 interleaves each code byte with a 0x43 byte: (q_b0 | 0x43 << 8), (q_b1 | 0x43 << 8)
        const uint32_t k43 = 0x43434343u;
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = {__builtin_amdgcn_perm(k43, lo, 0x04010400u), __builtin_amdgcn_perm(k43, lo, 0x04030402u),
                         __builtin_amdgcn_perm(k43, hi, 0x04010400u), __builtin_amdgcn_perm(k43, hi, 0x04030402u)};
        return __builtin_bit_cast(bf16x8, v);
    }
    __device__ static int x_first(int s, int half) { return half ? 16 + 4 * s : 4 * s; }
    // raw scale data of (row, block), and the block's coefficients (c1, c2)
    // from it: y += c1 * P + c2 * S
    __device__ static void load_scale(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K,
                                      int blk, uint32_t* r) {
        if constexpr (FMT == LW_Q4_0) {
            r[0] = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk));
        } else if constexpr (FMT == LW_Q4_1) {
            r[0] = *reinterpret_cast<const uint32_t*>(W + off1 + 4 * (row * (K / 32u) + (uint32_t)blk));
        } else {
            const uint64_t sb = row * (K / 256u) + (uint32_t)(blk >> 3);
            const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * sb);
            r[0] = rec[0];
            r[1] = rec[1];
            r[2] = rec[2];
            r[3] = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * sb);
        }
    }
    // raw scale data of the 8 blocks blk0 .. blk0+7 of a row (blk0 a multiple
    // of 8: one 16-byte load of d values, or one super-block's record and
    // {d, dmin}), and the coefficients of block blk0 + e from it
    __device__ static void load_scale8(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K,
                                       int blk0, uint32_t* r) {
        if constexpr (FMT == LW_Q4_0) {
            const uint4 v = *reinterpret_cast<const uint4*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk0));
            r[0] = v.x;
            r[1] = v.y;
            r[2] = v.z;
            r[3] = v.w;
        } else if constexpr (FMT == LW_Q4_1) {
            const uint4* p = reinterpret_cast<const uint4*>(W + off1 + 4 * (row * (K / 32u) + (uint32_t)blk0));
            const uint4 v = p[0], u = p[1];
            r[0] = v.x;
            r[1] = v.y;
            r[2] = v.z;
            r[3] = v.w;
            r[4] = u.x;
            r[5] = u.y;
            r[6] = u.z;
            r[7] = u.w;
        } else {
            load_scale(W, off1, off2, row, K, blk0, r);
        }
    }
    __device__ static void coef8(const uint32_t* r, int e, float* c1, float* c2) {
        if constexpr (FMT == LW_Q4_0) {
            const float d = half_bits_to_float((r[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
            *c1 = d;
            *c2 = -136.0f * d;
        } else if constexpr (FMT == LW_Q4_1) {
            coef_raw(r + e, e, c1, c2);
        } else {
            coef_raw(r, e, c1, c2);
        }
    }
    __device__ static void coef_raw(const uint32_t* r, int blk, float* c1, float* c2) {
        if constexpr (FMT == LW_Q4_0) {
            const float d = half_bits_to_float(r[0]);
            *c1 = d;
            *c2 = -136.0f * d;
        } else if constexpr (FMT == LW_Q4_1) {
            const float d = half_bits_to_float(r[0] & 0xFFFFu);
            *c1 = d;
            *c2 = __builtin_fmaf(-128.0f, d, half_bits_to_float(r[0] >> 16));  // m - 128 d
        } else {
            const uint32_t ts = 6u * (uint32_t)(blk & 7), tm = ts + 16u;
            const bool sl = ts < 32u, ml = tm < 32u;
            const uint32_t sc = __builtin_amdgcn_alignbit(sl ? r[1] : 0u, sl ? r[0] : r[1], ts & 31u) & 63u;
            const uint32_t m = __builtin_amdgcn_alignbit(ml ? r[2] : 0u, ml ? r[1] : r[2], tm & 31u) & 63u;
            const float ds = half_bits_to_float(r[3] & 0xFFFFu) * (float)sc;
            const float dm = half_bits_to_float(r[3] >> 16) * (float)m;
            *c1 = ds;
            *c2 = -__builtin_fmaf(128.0f, ds, dm);
        }
    }
};
template <>
struct MF<LW_Q4_0> : MF4<LW_Q4_0> {};
template <>
struct MF<LW_Q4_K> : MF4<LW_Q4_K> {};
template <>
struct MF<LW_Q4_1> : MF4<LW_Q4_1> {};
// The 5-bit formats share the 4-bit formats' scale data (read from their own
// planes, passed in the same argument slots), and the biased code 128 + q with
// q in [0, 31] is still an exact bfloat16: Q5_1 and Q5_K take Q4_1's and
// Q4_K's coefficients as they are; Q5_0 is w = d (q - 16), so 128 + q =
// (q - 16) + 144.
template <>
struct MF<LW_Q5_0> : MF4<LW_Q4_0> {
    __device__ static void coef8(const uint32_t* r, int e, float* c1, float* c2) {
        const float d = half_bits_to_float((r[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
        *c1 = d;
        *c2 = -144.0f * d;
    }
};
template <>
struct MF<LW_Q5_1> : MF4<LW_Q4_1> {};
template <>
struct MF<LW_Q5_K> : MF4<LW_Q4_K> {};
// The formats with 16-element sub-blocks: one coefficient pair per sub-block
// (one MFMA K-step), read for the 16 sub-blocks of 8 blocks (one super-block)
// at a time. Q6_K: w = d sc (q - 32), 6-bit q, signed 8-bit sc, so 128 + q =
// (q - 32) + 160. Q2_K: w = d sc q - dmin m, 2-bit q, 4-bit sc and m.
template <>
struct MF<LW_Q6_K> {
    static constexpr bool kSums = true;
    static constexpr int kRaw = 5;  // 16 scale bytes, then d
    __device__ static void load_scale16(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K,
                                        int blk0, uint32_t* r) {
        const uint4 v = *reinterpret_cast<const uint4*>(W + off1 + row * (K / 16u) + 2u * (uint32_t)blk0);
        r[0] = v.x;
        r[1] = v.y;
        r[2] = v.z;
        r[3] = v.w;
        r[4] = *reinterpret_cast<const uint16_t*>(W + off2 + 2u * (row * (K / 256u) + (uint32_t)(blk0 >> 3)));
    }
    __device__ static void coef16(const uint32_t* r, int u, float* c1, float* c2) {
        const float ds = half_bits_to_float(r[4]) * (float)sbyte_at(r[u >> 2], u & 3);  // exact
        *c1 = ds;
        *c2 = -160.0f * ds;  // exact
    }
    __device__ static int sbyte_at(uint32_t w, int i) { return (int)(int8_t)(uint8_t)(w >> (8 * i)); }
};
template <>
struct MF<LW_Q2_K> {
    static constexpr bool kSums = true;
    static constexpr int kRaw = 5;  // 16 {scale, min} bytes, then {d, dmin}
    __device__ static void load_scale16(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K,
                                        int blk0, uint32_t* r) {
        const uint4 v = *reinterpret_cast<const uint4*>(W + off1 + row * (K / 16u) + 2u * (uint32_t)blk0);
        r[0] = v.x;
        r[1] = v.y;
        r[2] = v.z;
        r[3] = v.w;
        r[4] = *reinterpret_cast<const uint32_t*>(W + off2 + 4u * (row * (K / 256u) + (uint32_t)(blk0 >> 3)));
    }
    __device__ static void coef16(const uint32_t* r, int u, float* c1, float* c2) {
        const uint32_t scm = (r[u >> 2] >> (8 * (u & 3))) & 0xFFu;
        const float ds = half_bits_to_float(r[4] & 0xFFFFu) * (float)(scm & 15u);  // exact
        const float dm = half_bits_to_float(r[4] >> 16) * (float)(scm >> 4);       // exact
        *c1 = ds;
        *c2 = -__builtin_fmaf(128.0f, ds, dm);
    }
};
// q1_0: w = +-d, the operand the exact bfloat16 +-1 of each bit; one d per
// 128 elements (4 blocks); no offset term.
template <>
struct MF<LW_Q1_0> {
    static constexpr bool kSums = false;
    static constexpr int kRaw = 1;  // the two binary16 d of 8 blocks
    __device__ static void load_scale8(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, int blk0,
                                       uint32_t* r) {
        r[0] = *reinterpret_cast<const uint32_t*>(W + off1 + 2u * (row * (K / 128u) + (uint32_t)(blk0 >> 2)));
    }
    __device__ static void coef8(const uint32_t* r, int e, float* c1, float* c2) {
        *c1 = half_bits_to_float((r[0] >> (16 * (e >> 2))) & 0xFFFFu);
        *c2 = 0.f;
    }
};
// MXFP4: the e2m1 values themselves are exact bfloat16 operands, so there is
// no offset term: y += 2^(E - 127) * P, with the block's e8m0 exponent E.
template <>
struct MF<LW_MXFP4> {
    static constexpr bool kSums = false;
    static constexpr int kRaw = 2;  // the 8 exponent bytes of 8 blocks
    __device__ static void load_scale8(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, int blk0,
                                       uint32_t* r) {
        const uint2 v = *reinterpret_cast<const uint2*>(W + off1 + row * (K / 32u) + (uint32_t)blk0);
        r[0] = v.x;
        r[1] = v.y;
    }
    __device__ static void coef8(const uint32_t* r, int e, float* c1, float* c2) {
        *c1 = e8m0_to_float((r[e >> 2] >> (8 * (e & 3))) & 0xFFu);
        *c2 = 0.f;
    }
};

template <>
struct MF<LW_Q8_0> {
    static constexpr bool kSums = false;
    static constexpr int kRaw = 4;  // raw scale words of 8 blocks
    // two words: elements 8s .. 8s+7; returned packed in one 64-bit value
    __device__ static uint64_t code_word(const uint8_t* W, uint64_t row, uint32_t K, int blk, int s) {
        return *reinterpret_cast<const uint64_t*>(W + row * K + 32u * (uint32_t)blk + 8u * s);
    }
    __device__ static bf16x8 decode(uint64_t w) {
        const uint32_t a = (uint32_t)w, b = (uint32_t)(w >> 32);
        bf16x8 v;
        v[0] = (__bf16)sbyte<0>(a);
        v[1] = (__bf16)sbyte<1>(a);
        v[2] = (__bf16)sbyte<2>(a);
        v[3] = (__bf16)sbyte<3>(a);
        v[4] = (__bf16)sbyte<0>(b);
        v[5] = (__bf16)sbyte<1>(b);
        v[6] = (__bf16)sbyte<2>(b);
        v[7] = (__bf16)sbyte<3>(b);
        return v;
    }
    __device__ static int x_first(int s, int half) { return 8 * s + 4 * half; }
    __device__ static void load_scale(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, int blk,
                                      uint32_t* r) {
        r[0] = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk));
    }
    __device__ static void coef_raw(const uint32_t* r, int, float* c1, float* c2) {
        *c1 = half_bits_to_float(r[0]);
        *c2 = 0.f;
    }
    __device__ static void load_scale8(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, int blk0,
                                       uint32_t* r) {
        const uint4 v = *reinterpret_cast<const uint4*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk0));
        r[0] = v.x;
        r[1] = v.y;
        r[2] = v.z;
        r[3] = v.w;
    }
    __device__ static void coef8(const uint32_t* r, int e, float* c1, float* c2) {
        *c1 = half_bits_to_float((r[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
        *c2 = 0.f;
    }
};

// Tiled kernel. A workgroup of WM waves computes BM = 64*WM weight rows x
// BN = 16*TT tokens over the blocks of one K split; wave wm owns rows
// 64*wm .. 64*wm+63 as four 16-row tiles rt and all BN tokens as TT tiles of
// 16. Roles in D = A . B: A is X (16 tokens x one 32-element block), B the
// decoded codes (one block x 16 weight rows), so lane l holds
// D[4*(l/16) + v][l % 16] = (token 4*(l/16) + v, weight row l % 16) and one
// coefficient per row tile and block serves all of a lane's outputs.
//
// A block's contribution has two parts. c1 * P: one FMA per output and block
// right after the block's MFMAs. c2 * S: a product over blocks,
// sum_b S[t][b] * c2[r][b], done on the matrix cores once per window of 16
// blocks (one v_mfma_f32_16x16x16_bf16 K-step spans the window), with S and
// c2 split three ways into bf16 parts (exact to 24 bits each): six partial
// products accumulated straight into the output tile.
//
// K advances in stages of kKB blocks. Per stage the workgroup converts the X
// slab (BN tokens x 32*kKB values) to hi/lo bf16 into one of two LDS stage
// buffers and appends the block sums S to the window buffer; the c1 and c2
// coefficients of a window's BM rows are computed once per window, one row
// per thread. Each wave loads the codes of its own 64 rows straight into
// registers, a quad of four blocks ahead. The vector work that bounds this
// kernel is the c1 FMAs, the code decode (amortized over the TT token tiles
// of a wave) and the X conversion (amortized over the BM rows of a
// workgroup); every address is a base computed once plus a stage offset.
//
// Work split: (row tile, token tile) pairs and, where those are too few to
// occupy every compute unit, K splits on super-block boundaries whose
// partial results are added to y atomically (y is zeroed first by a fill
// kernel). Consecutive workgroup indices go to different XCDs, so the tile
// order is permuted to give each XCD a contiguous run of tiles: the token
// tiles of a row tile then share that XCD's L2 for the weight tile.
constexpr int kKB = 2;    // blocks per stage
constexpr int kWin = 16;  // blocks per coefficient window (the c2 * S product: one 16x16x16 K-step)

template <int WM, int TT>
struct GemmTile {
    static constexpr int BM = 64 * WM, BN = 16 * TT, NT = 64 * WM;
    static constexpr int XI = kKB * BN * 4 / NT;  // X items (8 values) per thread and stage
    static_assert(XI >= 1 && XI * NT == kKB * BN * 4, "whole X items per thread");
    static constexpr int kX = kKB * 4 * BN;                // bf16x8 entries per half per stage
    static constexpr size_t kStage = (size_t)2 * kX * 16;  // xh, xl [kKB][4][BN]
    static constexpr size_t kC = (size_t)kWin * BM * 4;    // c1 (or c2) of a window
    static constexpr size_t kS = (size_t)kWin * BN * 4;    // block sums of a window
    static constexpr size_t bytes(bool sums) { return 2 * kStage + 2 * kC + (sums ? kC + 2 * kS : 0); }
};

// v = h + m + l with h, m, l bfloat16 (round to nearest even at each step):
// exact for any float whose significand fits 24 bits.
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void split3_bf16x4(const float* v, bf16x4* h, bf16x4* m, bf16x4* l) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    u32x2 hw, mw, lw;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const float a = v[2 * p], b = v[2 * p + 1];
        const uint32_t hb = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), bf16x2));
        const float ra = a - __builtin_bit_cast(float, hb << 16), rb = b - __builtin_bit_cast(float, hb & 0xFFFF0000u);
        const uint32_t mb = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{ra, rb}), bf16x2));
        const float qa = ra - __builtin_bit_cast(float, mb << 16), qb = rb - __builtin_bit_cast(float, mb & 0xFFFF0000u);
        hw[p] = hb;
        mw[p] = mb;
        lw[p] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{qa, qb}), bf16x2));
    }
    *h = __builtin_bit_cast(bf16x4, hw);
    *m = __builtin_bit_cast(bf16x4, mw);
    *l = __builtin_bit_cast(bf16x4, lw);
}

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

// 4 x 4 transpose across the four 16-lane groups: lane (g, i) holds the words
// w0..w3 of block g of its row; afterwards word j of the result is word g of
// block j (the slice of block j this lane feeds to the matrix core).
__device__ __forceinline__ u32x4v transpose_quad(u32x4v w) {
    const auto s02 = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
    const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    return u32x4v{s01[0], s01[1], s23[0], s23[1]};
}

template <int FMT, int WM, int TT>
__global__ void __launch_bounds__(64 * WM) __attribute__((amdgpu_waves_per_eu(2, 2)))
    gemm_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                int64_t K, int64_t N, int64_t off1, int64_t off2, GemmSplit sp) {
    using T = MF<FMT>;
    using TL = GemmTile<WM, TT>;
    constexpr int BM = TL::BM, BN = TL::BN, NT = TL::NT, XI = TL::XI;
    constexpr bool kQ4 = FMT != LW_Q8_0;
    constexpr bool kSums = T::kSums;
    extern __shared__ bf16x8 smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wm = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int i16 = lane & 15, s4 = lane >> 4;

    // tile of this workgroup: XCD x (= index mod 8) takes the contiguous run
    // of tiles [x * G/8, (x+1) * G/8) when G is a multiple of 8
    const int64_t G = (int64_t)gridDim.x;
    const int64_t bi = (int64_t)blockIdx.x;
    const int64_t L = (G & 7) == 0 ? (bi & 7) * (G >> 3) + (bi >> 3) : bi;
    const int64_t tt_i = L % sp.ntt;
    const int64_t rest = L / sp.ntt;
    const int split = (int)(rest % sp.ks);
    const int64_t rti = rest / sp.ks;
    const int64_t row0 = rti * BM;
    const int64_t tok0 = tt_i * BN;
    const uint32_t K32 = (uint32_t)K;
    const int nsb = (int)(K / 256);
    const int sb0 = split * sp.sbp;
    const int sb1 = sb0 + sp.sbp < nsb ? sb0 + sp.sbp : nsb;
    const int kb0 = 8 * sb0;            // first block of the split
    const int nb = 8 * (sb1 - sb0);     // blocks of the split (a multiple of 8)
    const int nst = nb / kKB;           // stages (a multiple of 4)
    const int nwin = (nb + kWin - 1) / kWin;

    char* lds = reinterpret_cast<char*>(smem);
    auto st_xh = [&](int bf) __attribute__((always_inline)) { return reinterpret_cast<bf16x8*>(lds + bf * TL::kStage); };
    auto st_xl = [&](int bf) __attribute__((always_inline)) { return st_xh(bf) + TL::kX; };
    auto win_c1 = [&](int w) __attribute__((always_inline)) {
        return reinterpret_cast<float*>(lds + 2 * TL::kStage + (w & 1) * TL::kC);
    };
    // c2 [row tile][g][row in tile][4]: lane (g, n) of a row tile reads the
    // c2 of blocks 4g..4g+3 of row n as one float4 (the 16x16x16 B operand);
    // S [token tile][g][token in tile][4] likewise (the A operand), one
    // buffer per window parity: the next window's sums are written while the
    // current window's product still reads its own
    float* win_c2 = reinterpret_cast<float*>(lds + 2 * TL::kStage + 2 * TL::kC);
    auto win_s = [&](int w) __attribute__((always_inline)) { return win_c2 + kWin * BM + (w & 1) * kWin * BN; };

    // ---- codes of this lane's rows (B operand columns), clamped; stores are masked ----
    const uint8_t* wp[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int64_t r = row0 + 64 * wm + 16 * rt + i16;
        const uint64_t rr = (uint64_t)(r < M ? r : M - 1);
        if constexpr (kQ4)
            wp[rt] = W + rr * (K32 / 2u) + 16u * (uint32_t)(kb0 + s4);
        else
            wp[rt] = W + rr * K32 + 32u * (uint32_t)kb0 + 8u * (uint32_t)s4;
    }
    // 4-bit formats: a quad = 4 blocks = 2 stages; lane (s4, i16) loads block
    // 4q + s4 of its row (16 bytes) and a register transpose hands it word s4
    // of each of the 4 blocks. Q8_0: per stage, word s4 of each block.
    u32x4v qraw[4], qcur[4];
    uint64_t cwA[4][kKB], cwB[4][kKB];
    auto load_quad = [&](int q) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) qraw[rt] = *reinterpret_cast<const u32x4v*>(wp[rt] + 64u * (uint32_t)q);
    };
    auto load_codes8 = [&](uint64_t (*cw)[kKB], int st) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int b = 0; b < kKB; ++b)
                cw[rt][b] = *reinterpret_cast<const uint64_t*>(wp[rt] + 32u * (uint32_t)(st * kKB + b));
    };

    // ---- window coefficients: thread tid handles row tid, all 16 blocks ----
    const int64_t crow = row0 + tid < M ? row0 + tid : M - 1;
    const int c_at = (tid >> 6) * 64 + (tid & 15) * 4 + ((tid >> 4) & 3);   // c1 slot (wave, row, rt) of this row
    float* const c2_row = win_c2 + (tid >> 4) * 256 + (tid & 15) * 4;       // + g * 64 + j
    uint32_t sraw[2][T::kRaw];
    auto load_win_scales = [&](int w) __attribute__((always_inline)) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            int blk0 = kb0 + w * kWin + 8 * h;
            blk0 = blk0 < kb0 + nb ? blk0 : kb0 + nb - 8;  // past the split: a valid copy, never used
            T::load_scale8(W, off1, off2, (uint64_t)crow, K32, blk0, sraw[h]);
        }
    };
    auto put_win_scales = [&](int w) __attribute__((always_inline)) {
        float* c1w = win_c1(w);
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int b16 = 8 * h + e;
                float c1, c2;
                T::coef8(sraw[h], e, &c1, &c2);
                c1w[b16 * BM + c_at] = c1;
                if constexpr (kSums) c2_row[(b16 >> 2) * 64 + (b16 & 3)] = c2;
            }
    };

    // ---- X stage producer: items (block b, token t, slice sl), fixed per thread ----
    const float* xp[XI];
    int xo[XI], so[XI], xb_[XI];
#pragma unroll
    for (int i = 0; i < XI; ++i) {
        const int it = tid + i * NT;
        const int sl = it & 3, t = (it >> 2) % BN, b = (it >> 2) / BN;
        // tokens past N read the last token: their outputs are never stored
        const int64_t tk = tok0 + t < N ? tok0 + t : N - 1;
        xp[i] = x + tk * K + 32 * (int64_t)(kb0 + b) + T::x_first(sl, 0);
        // token slots are XOR-swizzled by the slice so that the four slices
        // written by a lane quad fall into different LDS banks
        xo[i] = (b * 4 + sl) * BN + (t ^ (sl << 2));
        so[i] = ((t >> 4) * 4) * 64 + (t & 15) * 4;  // S slot of (t, block 0); + (b16 >> 2) * 64 + (b16 & 3)
        xb_[i] = b;
    }
    constexpr int kHalf2 = kQ4 ? 16 : 4;  // offset of the slice's second 4 values
    float4 xa[XI], xb[XI];
    auto fetch = [&](int st) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < XI; ++i) {
            const float* p = xp[i] + 32 * kKB * st;
            xa[i] = *reinterpret_cast<const float4*>(p);
            xb[i] = *reinterpret_cast<const float4*>(p + kHalf2);
        }
    };
    auto commit = [&](int bf, int st) __attribute__((always_inline)) {
        bf16x8* xh = st_xh(bf);
        bf16x8* xl = st_xl(bf);
#pragma unroll
        for (int i = 0; i < XI; ++i) {
            const float v[8] = {xa[i].x, xa[i].y, xa[i].z, xa[i].w, xb[i].x, xb[i].y, xb[i].z, xb[i].w};
            bf16x8 h, l;
            float sum = split_bf16x8(v, &h, &l);
            xh[xo[i]] = h;
            xl[xo[i]] = l;
            if constexpr (kSums) {
                const int b16 = (st * kKB + xb_[i]) % kWin;
                // the 4 slices of (block, token) are one lane quad: after two
                // exchanges every lane of it holds the block sum, and all four
                // store it (one address, one value; no branch in the stage)
                sum += dpp_move<0xB1>(sum);
                sum += dpp_move<0x4E>(sum);
                win_s(st * kKB / kWin)[so[i] + (b16 >> 2) * 64 + (b16 & 3)] = sum;
            }
        }
    };

    f32x4 acc[4][TT];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) acc[rt][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // A operand slot of token tile tt for this lane (block 0 of a stage)
    const int a_at = s4 * BN + (i16 ^ (s4 << 2));
    // stage st from LDS buffer bf; the codes of its block b: word j0 + b of
    // qcur (4-bit) or cw[.][b] (Q8_0)
    auto compute = [&](int bf, int st, int j0, uint64_t (*cw)[kKB]) __attribute__((always_inline)) {
        const bf16x8* xh = st_xh(bf);
        const bf16x8* xl = st_xl(bf);
        const float4* c1w = reinterpret_cast<const float4*>(win_c1(st * kKB / kWin));
        // A operands one token tile ahead (across the block boundary too):
        // the LDS reads of tile tt+1 are in flight during tile tt's MFMAs
        bf16x8 ahn = xh[a_at], aln = xl[a_at];
#pragma unroll
        for (int b = 0; b < kKB; ++b) {
            const int b16 = (st * kKB + b) % kWin;
            const float4 c1v = c1w[(b16 * BM + 64 * wm) / 4 + i16];
            const float c1[4] = {c1v.x, c1v.y, c1v.z, c1v.w};
            // the block's codes of the four row tiles, decoded once for all
            // token tiles
            bf16x8 bw[4];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                if constexpr (kQ4)
                    bw[rt] = T::decode(qcur[rt][j0 + b]);
                else
                    bw[rt] = T::decode(cw[rt][b]);
            }
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                const bf16x8 ah = ahn, al = aln;
                if (tt + 1 < TT) {
                    ahn = xh[b * 4 * BN + a_at + 16 * (tt + 1)];
                    aln = xl[b * 4 * BN + a_at + 16 * (tt + 1)];
                } else if (b + 1 < kKB) {
                    ahn = xh[(b + 1) * 4 * BN + a_at];
                    aln = xl[(b + 1) * 4 * BN + a_at];
                }
#pragma unroll
                for (int rt = 0; rt < 4; ++rt) {
                    f32x4 p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bw[rt], f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bw[rt], p, 0, 0, 0);
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[rt][tt][v] = __builtin_fmaf(c1[rt], p[v], acc[rt][tt][v]);
                }
            }
        }
    };
    // acc += S(window) . c2(window)^T for window w (nv valid blocks; S of the
    // others is masked to zero)
    auto bias = [&](int w) __attribute__((always_inline)) {
        const int nv = nb - w * kWin < kWin ? nb - w * kWin : kWin;
        bf16x4 sh[TT], sm[TT], sl[TT];
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
            const float4 s = reinterpret_cast<const float4*>(win_s(w))[(tt * 4 + s4) * 16 + i16];
            const float v[4] = {4 * s4 + 0 < nv ? s.x : 0.f, 4 * s4 + 1 < nv ? s.y : 0.f,
                                4 * s4 + 2 < nv ? s.z : 0.f, 4 * s4 + 3 < nv ? s.w : 0.f};
            split3_bf16x4(v, &sh[tt], &sm[tt], &sl[tt]);
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            const float4 c = reinterpret_cast<const float4*>(win_c2)[((wm * 4 + rt) * 4 + s4) * 16 + i16];
            const float v[4] = {c.x, c.y, c.z, c.w};
            bf16x4 chh, chm, chl;
            split3_bf16x4(v, &chh, &chm, &chl);
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                f32x4 a = acc[rt][tt];
                a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sh[tt], chh, a, 0, 0, 0);
                a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sh[tt], chm, a, 0, 0, 0);
                a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sm[tt], chh, a, 0, 0, 0);
                a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sh[tt], chl, a, 0, 0, 0);
                a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sm[tt], chm, a, 0, 0, 0);
                a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sl[tt], chh, a, 0, 0, 0);
                acc[rt][tt] = a;
            }
        }
    };
    // the FMAs of the stage complete before the window's branch: sunk past
    // it they would keep every partial product of the stage live across it
    auto pin = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) asm volatile("" : "+v"(acc[rt][tt]));
    };
    // after stage st: when it ends a window, the window's c2 * S product is
    // added, and (after a barrier: the window buffers are reused) the next
    // window's coefficients are stored and the one after is prefetched
    auto window_end = [&](int st) __attribute__((always_inline)) {
        if (((st + 1) * kKB) % kWin == 0 || st == nst - 1) {
            const int w = st * kKB / kWin;
            if constexpr (kSums) bias(w);
            __syncthreads();
            if (w + 1 < nwin) put_win_scales(w + 1);
            load_win_scales(w + 2 < nwin ? w + 2 : nwin - 1);
        }
    };

    // ---- prologue ----
    if constexpr (kQ4) {
        load_quad(0);
    } else {
        load_codes8(cwA, 0);
        load_codes8(cwB, 1);
    }
    load_win_scales(0);
    fetch(0);
    put_win_scales(0);
    load_win_scales(nwin > 1 ? 1 : 0);
    commit(0, 0);
    fetch(1);
    __syncthreads();

    // ---- main loop: stages in pairs (one quad of blocks); all global loads
    // are unconditional (indices past the end are clamped; those copies are
    // never used), so the compiler counts them and prefetches stay in flight
    for (int st = 0; st < nst; st += 2) {
        const int s2 = st + 2 < nst ? st + 2 : nst - 1;
        const int s3 = st + 3 < nst ? st + 3 : nst - 1;
        if constexpr (kQ4) {
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) qcur[rt] = transpose_quad(qraw[rt]);
            load_quad(s2 / 2);
        }
        // the next stage's X conversion shares a basic block with this
        // stage's MFMAs, so its vector work can issue while they run
        compute(0, st, 0, cwA);
        if constexpr (!kQ4) load_codes8(cwA, s2);
        commit(1, st + 1);
        fetch(s2);
        pin();
        window_end(st);
        __syncthreads();
        compute(1, st + 1, 2, cwB);
        if constexpr (!kQ4) load_codes8(cwB, s3);
        commit(0, s2);  // past the end: a copy of the last stage, never read
        fetch(s3);
        pin();
        window_end(st + 1);
        __syncthreads();
    }

    // store: lane holds tokens 16*tt + 4*s4 + v of weight row 64*wm + 16*rt + i16
    // (K splits: added to the zeroed y)
    const bool split_k = sp.ks > 1;
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int64_t r = row0 + 64 * wm + 16 * rt + i16;
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t t = tok0 + 16 * tt + 4 * s4 + v;
                if (r < M && t < N) {
                    float* const o = y + t * M + r;
                    if (split_k)
                        unsafeAtomicAdd(o, acc[rt][tt][v]);
                    else
                        *o = acc[rt][tt][v];
                }
            }
    }
}

// ---------------------------------------------------------------------------
// The 4-bit formats on 32 x 32 output tiles (v_mfma_f32_32x32x16_bf16, which
// runs at about twice the rate of the 16 x 16 x 32 form on MI355X: 2.2-2.4
// against 0.9-1.4 dense bf16 PFLOP/s in a throughput probe). Operand layout
// (verified on the GPU): lane l supplies A[l % 32][8 (l / 32) + v] and
// B[8 (l / 32) + v][l % 32], v = 0..7, and receives D[i][l % 32] for
// i = 8 (v / 4) + 4 (l / 32) + v % 4, v = 0..15. A is X (32 tokens x 16 k),
// B the biased codes (16 k x 32 weight rows): a lane holds 16 tokens of one
// weight row, so one c1 per lane and tile scales all of its outputs.
//
// A 32-element block is two K-steps: lane (h, n) feeds elements 8h .. 8h+7
// (K-step 0) and 16 + 8h .. 16 + 8h + 7 (K-step 1) of the block, which are the
// low and the high nibbles of the block's bytes 8h .. 8h+7. Per block and
// tile: four MFMAs (two K-steps, X high and low parts), then the 16 c1 FMAs.
// A workgroup of WM waves covers 64 WM rows x 64 tokens; each wave owns 64
// rows x 64 tokens as 2 x 2 tiles. The rest (stages, windows of 16 blocks
// for the c2 * S product, now on v_mfma_f32_32x32x8_bf16, K splits and the
// XCD-grouped tile order) is as in gemm_kernel.
template <int WM>
struct Tile32 {
    static constexpr int BM = 64 * WM, BN = 64, NT = 64 * WM;
    static constexpr int XI = kKB * BN * 4 / NT;  // X items (8 values) per thread and stage
    static_assert(XI >= 1 && XI * NT == kKB * BN * 4, "whole X items per thread");
    static constexpr int kX = kKB * 4 * BN;                // bf16x8 entries per half per stage: [b][2s+h][t]
    static constexpr size_t kStage = (size_t)2 * kX * 16;  // xh, xl
    static constexpr size_t kC = (size_t)kWin * BM * 4;    // c1 (or c2) of a window
    static constexpr size_t kS = (size_t)kWin * BN * 4;    // block sums of a window
    static constexpr size_t bytes() { return 2 * kStage + 2 * kC + kC + 2 * kS; }
};

// Biased bf16 codes (bits 0x4300 | q) of bytes 8h .. 8h+7 of a block, given as
// two words: the low nibbles feed K-step 0, the high nibbles K-step 1.
__device__ __forceinline__ void decode8(uint32_t w0, uint32_t w1, bf16x8* s0, bf16x8* s1) {
    const uint32_t k43 = 0x43434343u;
    const uint32_t l0 = opaque(w0 & 0x0F0F0F0Fu), l1 = opaque(w1 & 0x0F0F0F0Fu);
    const uint32_t h0 = opaque((w0 >> 4) & 0x0F0F0F0Fu), h1 = opaque((w1 >> 4) & 0x0F0F0F0Fu);
    const u32x4v a = {__builtin_amdgcn_perm(k43, l0, 0x04010400u), __builtin_amdgcn_perm(k43, l0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, l1, 0x04010400u), __builtin_amdgcn_perm(k43, l1, 0x04030402u)};
    const u32x4v b = {__builtin_amdgcn_perm(k43, h0, 0x04010400u), __builtin_amdgcn_perm(k43, h0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, h1, 0x04010400u), __builtin_amdgcn_perm(k43, h1, 0x04030402u)};
    *s0 = __builtin_bit_cast(bf16x8, a);
    *s1 = __builtin_bit_cast(bf16x8, b);
}

// The 5-bit formats: as decode8, with the fifth bits of the 16 elements
// merged in first (spread4). hb holds them in element order: bits 0-7 for
// elements 8h .. 8h+7 (K-step 0), bits 8-15 for 16 + 8h .. 16 + 8h + 7
// (K-step 1).
__device__ __forceinline__ void decode8_q5(uint32_t w0, uint32_t w1, uint32_t hb, bf16x8* s0, bf16x8* s1) {
    const uint32_t k43 = 0x43434343u;
    const uint32_t l0 = opaque((w0 & 0x0F0F0F0Fu) | spread4((hb << 4) & 0xF0u));
    const uint32_t l1 = opaque((w1 & 0x0F0F0F0Fu) | spread4(hb & 0xF0u));
    const uint32_t h0 = opaque(((w0 >> 4) & 0x0F0F0F0Fu) | spread4((hb >> 4) & 0xF0u));
    const uint32_t h1 = opaque(((w1 >> 4) & 0x0F0F0F0Fu) | spread4((hb >> 8) & 0xF0u));
    const u32x4v a = {__builtin_amdgcn_perm(k43, l0, 0x04010400u), __builtin_amdgcn_perm(k43, l0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, l1, 0x04010400u), __builtin_amdgcn_perm(k43, l1, 0x04030402u)};
    const u32x4v b = {__builtin_amdgcn_perm(k43, h0, 0x04010400u), __builtin_amdgcn_perm(k43, h0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, h1, 0x04010400u), __builtin_amdgcn_perm(k43, h1, 0x04030402u)};
    *s0 = __builtin_bit_cast(bf16x8, a);
    *s1 = __builtin_bit_cast(bf16x8, b);
}

// Q6_K: as decode8, with the two high bits of the 16 elements merged in. hw
// holds them in element order, two bits each: bits 0-15 for elements 8h ..
// 8h+7 (K-step 0), bits 16-31 for 16 + 8h .. 16 + 8h + 7 (K-step 1).
__device__ __forceinline__ void decode8_q6(uint32_t w0, uint32_t w1, uint32_t hw, bf16x8* s0, bf16x8* s1) {
    const uint32_t k43 = 0x43434343u;
    const uint32_t l0 = opaque((w0 & 0x0F0F0F0Fu) | spread2_hi(hw & 0xFFu));
    const uint32_t l1 = opaque((w1 & 0x0F0F0F0Fu) | spread2_hi((hw >> 8) & 0xFFu));
    const uint32_t h0 = opaque(((w0 >> 4) & 0x0F0F0F0Fu) | spread2_hi((hw >> 16) & 0xFFu));
    const uint32_t h1 = opaque(((w1 >> 4) & 0x0F0F0F0Fu) | spread2_hi(hw >> 24));
    const u32x4v a = {__builtin_amdgcn_perm(k43, l0, 0x04010400u), __builtin_amdgcn_perm(k43, l0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, l1, 0x04010400u), __builtin_amdgcn_perm(k43, l1, 0x04030402u)};
    const u32x4v b = {__builtin_amdgcn_perm(k43, h0, 0x04010400u), __builtin_amdgcn_perm(k43, h0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, h1, 0x04010400u), __builtin_amdgcn_perm(k43, h1, 0x04030402u)};
    *s0 = __builtin_bit_cast(bf16x8, a);
    *s1 = __builtin_bit_cast(bf16x8, b);
}
// Q2_K: the 2-bit codes alone, in the same layout as decode8_q6's hw.
__device__ __forceinline__ void decode8_q2(uint32_t hw, bf16x8* s0, bf16x8* s1) {
    const uint32_t k43 = 0x43434343u;
    const uint32_t l0 = opaque(spread2_lo(hw & 0xFFu));
    const uint32_t l1 = opaque(spread2_lo((hw >> 8) & 0xFFu));
    const uint32_t h0 = opaque(spread2_lo((hw >> 16) & 0xFFu));
    const uint32_t h1 = opaque(spread2_lo(hw >> 24));
    const u32x4v a = {__builtin_amdgcn_perm(k43, l0, 0x04010400u), __builtin_amdgcn_perm(k43, l0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, l1, 0x04010400u), __builtin_amdgcn_perm(k43, l1, 0x04030402u)};
    const u32x4v b = {__builtin_amdgcn_perm(k43, h0, 0x04010400u), __builtin_amdgcn_perm(k43, h0, 0x04030402u),
                      __builtin_amdgcn_perm(k43, h1, 0x04010400u), __builtin_amdgcn_perm(k43, h1, 0x04030402u)};
    *s0 = __builtin_bit_cast(bf16x8, a);
    *s1 = __builtin_bit_cast(bf16x8, b);
}

// q1_0: the 16 bits hb (as decode8_q5's) as bfloat16 +-1.
__device__ __forceinline__ void decode8_q1(uint32_t hb, bf16x8* s0, bf16x8* s1) {
    uint32_t a[4], b[4];
    sign_pairs(hb & 15u, &a[0], &a[1]);
    sign_pairs((hb >> 4) & 15u, &a[2], &a[3]);
    sign_pairs((hb >> 8) & 15u, &b[0], &b[1]);
    sign_pairs((hb >> 12) & 15u, &b[2], &b[3]);
    *s0 = __builtin_bit_cast(bf16x8, (u32x4v{a[0], a[1], a[2], a[3]}));
    *s1 = __builtin_bit_cast(bf16x8, (u32x4v{b[0], b[1], b[2], b[3]}));
}

// MXFP4: both K-steps through fp4_pairs (lw_device.hpp).
__device__ __forceinline__ void decode8_fp4(uint32_t w0, uint32_t w1, bf16x8* s0, bf16x8* s1) {
    uint32_t a[4], b[4];
    fp4_pairs(opaque(w0 & 0x07070707u), (w0 << 4) & 0x80808080u, &a[0], &a[1]);
    fp4_pairs(opaque(w1 & 0x07070707u), (w1 << 4) & 0x80808080u, &a[2], &a[3]);
    fp4_pairs(opaque((w0 >> 4) & 0x07070707u), w0 & 0x80808080u, &b[0], &b[1]);
    fp4_pairs(opaque((w1 >> 4) & 0x07070707u), w1 & 0x80808080u, &b[2], &b[3]);
    *s0 = __builtin_bit_cast(bf16x8, (u32x4v{a[0], a[1], a[2], a[3]}));
    *s1 = __builtin_bit_cast(bf16x8, (u32x4v{b[0], b[1], b[2], b[3]}));
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int FMT, int WM>
__global__ void __launch_bounds__(64 * WM) __attribute__((amdgpu_waves_per_eu(2, 2)))
    gemm32_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                  int64_t K, int64_t N, int64_t off1, int64_t off2, int64_t offh, GemmSplit sp) {
    using T = MF<FMT>;
    using TL = Tile32<WM>;
    constexpr int BM = TL::BM, BN = TL::BN, NT = TL::NT, XI = TL::XI;
    constexpr bool kQ5 = FMT == LW_Q5_0 || FMT == LW_Q5_1 || FMT == LW_Q5_K;
    constexpr bool kFp4 = FMT == LW_MXFP4;
    constexpr bool kQ6 = FMT == LW_Q6_K, kQ2 = FMT == LW_Q2_K;
    constexpr bool kQ1 = FMT == LW_Q1_0;  // its 1-bit plane is laid out as the fifth-bit planes
    constexpr bool kSub16 = kQ6 || kQ2;  // one coefficient pair per 16-element K-step
    // a window holds kWin coefficient units: blocks, or the sub-blocks of kWin / 2 blocks
    constexpr int KWB = kSub16 ? kWin / 2 : kWin;
    static_assert(FMT != LW_Q8_0 && (T::kSums || kFp4 || kQ1), "the formats with 32-element K-steps of bf16 codes");
    extern __shared__ bf16x8 smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wm = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n32 = lane & 31, h = lane >> 5;

    // tile of this workgroup (XCD-grouped order, as in gemm_kernel)
    const int64_t G = (int64_t)gridDim.x;
    const int64_t bi = (int64_t)blockIdx.x;
    const int64_t L = (G & 7) == 0 ? (bi & 7) * (G >> 3) + (bi >> 3) : bi;
    const int64_t tt_i = L % sp.ntt;
    const int64_t rest = L / sp.ntt;
    const int split = (int)(rest % sp.ks);
    const int64_t rti = rest / sp.ks;
    const int64_t row0 = rti * BM;
    const int64_t tok0 = tt_i * BN;
    const uint32_t K32 = (uint32_t)K;
    const int nsb = (int)(K / 256);
    const int sb0 = split * sp.sbp;
    const int sb1 = sb0 + sp.sbp < nsb ? sb0 + sp.sbp : nsb;
    const int kb0 = 8 * sb0;
    const int nb = 8 * (sb1 - sb0);
    const int nst = nb / kKB;
    const int nwin = (nb + KWB - 1) / KWB;

    char* lds = reinterpret_cast<char*>(smem);
    auto st_xh = [&](int bf) __attribute__((always_inline)) { return reinterpret_cast<bf16x8*>(lds + bf * TL::kStage); };
    auto st_xl = [&](int bf) __attribute__((always_inline)) { return st_xh(bf) + TL::kX; };
    auto win_c1 = [&](int w) __attribute__((always_inline)) {
        return reinterpret_cast<float*>(lds + 2 * TL::kStage + (w & 1) * TL::kC);
    };
    // c2 [row tile of 32][k-group g = block / 4][row in tile][4] and S
    // [k-group][token][4] (one buffer per window parity): the operands of
    // v_mfma_f32_32x32x8_bf16, lane (h, n) reading one float4 of each
    float* win_c2 = reinterpret_cast<float*>(lds + 2 * TL::kStage + 2 * TL::kC);
    auto win_s = [&](int w) __attribute__((always_inline)) { return win_c2 + kWin * BM + (w & 1) * kWin * BN; };

    // ---- codes: lane (h, n) of row tile rt reads row 64 wm + 32 rt + n, bytes
    // [32h, 32h + 32) of each quad's 64 (blocks 2h, 2h + 1) ----
    const uint8_t* wp[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        const int64_t r = row0 + 64 * wm + 32 * rt + n32;
        const uint64_t rr = (uint64_t)(r < M ? r : M - 1);
        wp[rt] = W + rr * (K32 / 2u) + 16u * (uint32_t)kb0 + 32u * (uint32_t)h;
    }
    u32x4v qraw[2][2], qcur[2][2];
    // the 5-bit formats: the quad's 16 bytes of fifth bits of the lane's row
    // (4 per block, byte j of a block for its elements 8j .. 8j+7)
    // the 2-bit planes (Q6_K high bits, Q2_K codes): 8 bytes per block, lane
    // (h, n) reads blocks 2h, 2h + 1 of the quad (16 bytes)
    const uint8_t* hp[2];
    u32x4v hraw[2];
    uint32_t hcur[2][kSub16 ? 4 : 2];
    if constexpr (kQ5 || kQ1 || kSub16) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            const int64_t r = row0 + 64 * wm + 32 * rt + n32;
            const uint64_t rr = (uint64_t)(r < M ? r : M - 1);
            if constexpr (kQ5 || kQ1)
                hp[rt] = W + offh + rr * (K32 / 8u) + 4u * (uint32_t)kb0;
            else
                hp[rt] = W + offh + rr * (K32 / 4u) + 8u * (uint32_t)kb0 + 16u * (uint32_t)h;
        }
    }
    auto load_quad = [&](int q) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            if constexpr (!kQ2 && !kQ1) {
                qraw[rt][0] = *reinterpret_cast<const u32x4v*>(wp[rt] + 64u * (uint32_t)q);
                qraw[rt][1] = *reinterpret_cast<const u32x4v*>(wp[rt] + 64u * (uint32_t)q + 16u);
            }
            if constexpr (kQ5 || kQ1) hraw[rt] = *reinterpret_cast<const u32x4v*>(hp[rt] + 16u * (uint32_t)q);
            if constexpr (kSub16) hraw[rt] = *reinterpret_cast<const u32x4v*>(hp[rt] + 32u * (uint32_t)q);
        }
    };
    // lanes 0-31 hold blocks 0, 1 of the quad and lanes 32-63 blocks 2, 3 (four
    // words each); swapping words 2, 3 of each low block with words 0, 1 of
    // each high block leaves every lane the two words it feeds of every block:
    // block 0 in words (0, 1) of qcur[0], block 1 in (0, 1) of qcur[1],
    // block 2 in (2, 3) of qcur[0], block 3 in (2, 3) of qcur[1]
    auto swap_quad = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int hv = 0; hv < (kQ2 || kQ1 ? 0 : 2); ++hv) {
                const u32x4v v = qraw[rt][hv];
                const auto s02 = __builtin_amdgcn_permlane32_swap(v[0], v[2], false, false);
                const auto s13 = __builtin_amdgcn_permlane32_swap(v[1], v[3], false, false);
                qcur[rt][hv] = u32x4v{s02[0], s13[0], s02[1], s13[1]};
            }
        // fifth bits (q1_0: the code bits): bytes h and 2 + h of each block's
        // word (the lane's elements of K-steps 0 and 1), two blocks per word
        if constexpr (kQ5 || kQ1) {
            const uint32_t hsel = 0x06040200u + 0x01010101u * (uint32_t)h;
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                hcur[rt][0] = __builtin_amdgcn_perm(hraw[rt][1], hraw[rt][0], hsel);
                hcur[rt][1] = __builtin_amdgcn_perm(hraw[rt][3], hraw[rt][2], hsel);
            }
        }
        // 2-bit planes: block k of the lane's pair as words (w0, w1) = bytes
        // 0-3, 4-7; lanes of half h need bytes 2h, 2h+1 of each (elements 8h ..
        // 8h+7 and 16 + 8h .. 16 + 8h + 7). Each lane packs the bytes the
        // lower half needs (0, 1, 4, 5) and those the upper half needs (2, 3,
        // 6, 7) of its own block k; one swap across the halves then leaves
        // every lane its bytes of block k and of block 2 + k.
        if constexpr (kSub16) {
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    const uint32_t w0 = hraw[rt][2 * k], w1 = hraw[rt][2 * k + 1];
                    const uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x05040100u);
                    const uint32_t hi = __builtin_amdgcn_perm(w1, w0, 0x07060302u);
                    const auto r = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
                    hcur[rt][k] = r[0];
                    hcur[rt][2 + k] = r[1];
                }
        }
    };

    // ---- window coefficients: thread tid handles row tid, all 16 blocks ----
    const int64_t crow = row0 + tid < M ? row0 + tid : M - 1;
    const int c_at = (tid >> 6) * 64 + (tid & 31) * 2 + ((tid >> 5) & 1);  // c1 slot of this row
    float* const c2_row = win_c2 + (tid >> 5) * 512 + (tid & 31) * 4;      // + g * 128 + j
    uint32_t sraw[2][T::kRaw];
    auto load_win_scales = [&](int w) __attribute__((always_inline)) {
#pragma unroll
        for (int hh = 0; hh < (kSub16 ? 1 : 2); ++hh) {
            int blk0 = kb0 + w * KWB + 8 * hh;
            blk0 = blk0 < kb0 + nb ? blk0 : kb0 + nb - 8;  // past the split: a valid copy, never used
            if constexpr (kSub16)
                T::load_scale16(W, off1, off2, (uint64_t)crow, K32, blk0, sraw[hh]);
            else
                T::load_scale8(W, off1, off2, (uint64_t)crow, K32, blk0, sraw[hh]);
        }
    };
    auto put_win_scales = [&](int w) __attribute__((always_inline)) {
        float* c1w = win_c1(w);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int b16 = 8 * hh + e;  // coefficient unit of the window
                float c1, c2;
                if constexpr (kSub16)
                    T::coef16(sraw[0], b16, &c1, &c2);
                else
                    T::coef8(sraw[hh], e, &c1, &c2);
                c1w[b16 * BM + c_at] = c1;
                if constexpr (T::kSums) c2_row[(b16 >> 2) * 128 + (b16 & 3)] = c2;
            }
    };

    // ---- X stage producer: item (block b, token t, quarter q = 2s + hx):
    // elements 16s + 8hx .. +7 of the block for token t ----
    const float* xp[XI];
    int xo[XI], so[XI], xb_[XI], xs_[XI];
#pragma unroll
    for (int i = 0; i < XI; ++i) {
        const int it = tid + i * NT;
        const int q = it & 3, t = (it >> 2) % BN, b = (it >> 2) / BN;
        const int64_t tk = tok0 + t < N ? tok0 + t : N - 1;  // past N: the last token, never stored
        xp[i] = x + tk * K + 32 * (int64_t)(kb0 + b) + 8 * q;
        xo[i] = (b * 4 + q) * BN + (t ^ (q << 2));  // the four quarters of a token in four bank groups
        so[i] = t * 4;                               // S slot of (t, unit 0); + (u >> 2) * 4 BN + (u & 3)
        xb_[i] = b;
        xs_[i] = q >> 1;                             // the K-step (sub-block) of the quarter
    }
    float4 xa[XI], xb[XI];
    auto fetch = [&](int st) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < XI; ++i) {
            const float* p = xp[i] + 32 * kKB * st;
            xa[i] = *reinterpret_cast<const float4*>(p);
            xb[i] = *reinterpret_cast<const float4*>(p + 4);
        }
    };
    auto commit = [&](int bf, int st) __attribute__((always_inline)) {
        bf16x8* xh = st_xh(bf);
        bf16x8* xl = st_xl(bf);
#pragma unroll
        for (int i = 0; i < XI; ++i) {
            const float v[8] = {xa[i].x, xa[i].y, xa[i].z, xa[i].w, xb[i].x, xb[i].y, xb[i].z, xb[i].w};
            bf16x8 hv, lv;
            float sum = split_bf16x8(v, &hv, &lv);
            xh[xo[i]] = hv;
            xl[xo[i]] = lv;
            if constexpr (kSub16) {
                // quarters 2s, 2s + 1 of (block, token) are a lane pair: one
                // exchange gives both the sum of sub-block s; both store it
                const int u = 2 * ((st * kKB + xb_[i]) % KWB) + xs_[i];
                sum += dpp_move<0xB1>(sum);
                win_s(st * kKB / KWB)[so[i] + (u >> 2) * 4 * BN + (u & 3)] = sum;
            } else if constexpr (T::kSums) {
                // the 4 quarters of (block, token) are one lane quad: after two
                // exchanges every lane holds the block sum; all four store it
                const int b16 = (st * kKB + xb_[i]) % kWin;
                sum += dpp_move<0xB1>(sum);
                sum += dpp_move<0x4E>(sum);
                win_s(st * kKB / kWin)[so[i] + (b16 >> 2) * 4 * BN + (b16 & 3)] = sum;
            }
        }
    };

    f32x16 acc[2][2];  // [row tile][token tile]
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[rt][tt][v] = 0.f;

    // A operand slot of K-step s (block 0 of a stage, token tile 0)
    int a_at[2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) a_at[s2] = (2 * s2 + h) * BN + (n32 ^ ((2 * s2 + h) << 2));
    // the words this lane feeds of quad block jb of row tile rt
    auto pair_of = [&](int rt, int jb, uint32_t* w0, uint32_t* w1) __attribute__((always_inline)) {
        const u32x4v v = qcur[rt][jb & 1];
        *w0 = jb < 2 ? v[0] : v[2];
        *w1 = jb < 2 ? v[1] : v[3];
    };
    auto compute = [&](int bf, int st, int j0) __attribute__((always_inline)) {
        const bf16x8* xh = st_xh(bf);
        const bf16x8* xl = st_xl(bf);
        const float2* c1w = reinterpret_cast<const float2*>(win_c1(st * kKB / KWB));
        // A operands one token tile ahead (across the block boundary too)
        bf16x8 an[2][2];  // [s][hi, lo]
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            an[s2][0] = xh[a_at[s2]];
            an[s2][1] = xl[a_at[s2]];
        }
#pragma unroll
        for (int b = 0; b < kKB; ++b) {
            const int b16 = (st * kKB + b) % KWB;
            // c1 of K-step 0 (the block's, or its first sub-block's) and, with
            // 16-element sub-blocks, c1b of K-step 1; [rt]
            float c1[2], c1b[2];
            {
                const int u0 = kSub16 ? 2 * b16 : b16;
                const float2 c1v = c1w[(u0 * BM + 64 * wm) / 2 + n32];
                c1[0] = c1v.x;
                c1[1] = c1v.y;
                if constexpr (kSub16) {
                    const float2 c1u = c1w[((u0 + 1) * BM + 64 * wm) / 2 + n32];
                    c1b[0] = c1u.x;
                    c1b[1] = c1u.y;
                }
            }
            bf16x8 bw[2][2];  // [rt][s]
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                uint32_t w0 = 0, w1 = 0;
                if constexpr (!kQ2 && !kQ1) pair_of(rt, j0 + b, &w0, &w1);
                if constexpr (kQ1) {
                    const int jb = j0 + b;
                    decode8_q1((hcur[rt][jb >> 1] >> (16 * (jb & 1))) & 0xFFFFu, &bw[rt][0], &bw[rt][1]);
                } else if constexpr (kQ5) {
                    const int jb = j0 + b;
                    decode8_q5(w0, w1, (hcur[rt][jb >> 1] >> (16 * (jb & 1))) & 0xFFFFu, &bw[rt][0], &bw[rt][1]);
                } else if constexpr (kQ6) {
                    decode8_q6(w0, w1, hcur[rt][j0 + b], &bw[rt][0], &bw[rt][1]);
                } else if constexpr (kQ2) {
                    decode8_q2(hcur[rt][j0 + b], &bw[rt][0], &bw[rt][1]);
                } else if constexpr (kFp4) {
                    decode8_fp4(w0, w1, &bw[rt][0], &bw[rt][1]);
                } else {
                    decode8(w0, w1, &bw[rt][0], &bw[rt][1]);
                }
            }
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) {
                bf16x8 a[2][2];
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    a[s2][0] = an[s2][0];
                    a[s2][1] = an[s2][1];
                }
                if (tt == 0) {
#pragma unroll
                    for (int s2 = 0; s2 < 2; ++s2) {
                        an[s2][0] = xh[b * 4 * BN + a_at[s2] + 32];
                        an[s2][1] = xl[b * 4 * BN + a_at[s2] + 32];
                    }
                } else if (b + 1 < kKB) {
#pragma unroll
                    for (int s2 = 0; s2 < 2; ++s2) {
                        an[s2][0] = xh[(b + 1) * 4 * BN + a_at[s2]];
                        an[s2][1] = xl[(b + 1) * 4 * BN + a_at[s2]];
                    }
                }
#pragma unroll
                for (int rt = 0; rt < 2; ++rt) {
                    f32x16 pz;
#pragma unroll
                    for (int v = 0; v < 16; ++v) pz[v] = 0.f;
                    f32x16 p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0][0], bw[rt][0], pz, 0, 0, 0);
                    p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0][1], bw[rt][0], p, 0, 0, 0);
                    if constexpr (kSub16) {
                        // each K-step is a sub-block with its own scale
#pragma unroll
                        for (int v = 0; v < 16; ++v) acc[rt][tt][v] = __builtin_fmaf(c1[rt], p[v], acc[rt][tt][v]);
                        p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1][0], bw[rt][1], pz, 0, 0, 0);
                        p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1][1], bw[rt][1], p, 0, 0, 0);
#pragma unroll
                        for (int v = 0; v < 16; ++v) acc[rt][tt][v] = __builtin_fmaf(c1b[rt], p[v], acc[rt][tt][v]);
                    } else {
                        p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1][0], bw[rt][1], p, 0, 0, 0);
                        p = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1][1], bw[rt][1], p, 0, 0, 0);
#pragma unroll
                        for (int v = 0; v < 16; ++v) acc[rt][tt][v] = __builtin_fmaf(c1[rt], p[v], acc[rt][tt][v]);
                    }
                }
            }
        }
    };
    // acc += S(window) . c2(window)^T for window w: two K-steps of 8 blocks on
    // v_mfma_f32_32x32x8_bf16, S and c2 split three ways into bf16 parts
    // (blocks past the split's end: S masked to zero); none without offsets
    auto bias = [&](int w) __attribute__((always_inline)) {
        if constexpr (!T::kSums) return;
        const int nvb = nb - w * KWB < KWB ? nb - w * KWB : KWB;  // valid blocks of the window
        const int nv = kSub16 ? 2 * nvb : nvb;                    // valid coefficient units
        const float4* sw = reinterpret_cast<const float4*>(win_s(w));
        const float4* cw = reinterpret_cast<const float4*>(win_c2);
#pragma unroll
        for (int s8 = 0; s8 < 2; ++s8) {
            const int g = 2 * s8 + h;  // k-group of this lane: blocks 4g .. 4g+3
            bf16x4 sh[2], sm[2], sl[2];
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) {
                const float4 sv = sw[g * BN + 32 * tt + n32];
                const float v[4] = {4 * g + 0 < nv ? sv.x : 0.f, 4 * g + 1 < nv ? sv.y : 0.f,
                                    4 * g + 2 < nv ? sv.z : 0.f, 4 * g + 3 < nv ? sv.w : 0.f};
                split3_bf16x4(v, &sh[tt], &sm[tt], &sl[tt]);
            }
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const float4 cv = cw[((wm * 2 + rt) * 4 + g) * 32 + n32];
                const float v[4] = {cv.x, cv.y, cv.z, cv.w};
                bf16x4 chh, chm, chl;
                split3_bf16x4(v, &chh, &chm, &chl);
#pragma unroll
                for (int tt = 0; tt < 2; ++tt) {
                    f32x16 a = acc[rt][tt];
                    a = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(sh[tt], chh, a, 0, 0, 0);
                    a = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(sh[tt], chm, a, 0, 0, 0);
                    a = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(sm[tt], chh, a, 0, 0, 0);
                    a = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(sh[tt], chl, a, 0, 0, 0);
                    a = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(sm[tt], chm, a, 0, 0, 0);
                    a = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(sl[tt], chh, a, 0, 0, 0);
                    acc[rt][tt] = a;
                }
            }
        }
    };
    auto pin = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) asm volatile("" : "+v"(acc[rt][tt]));
    };
    auto window_end = [&](int st) __attribute__((always_inline)) {
        if (((st + 1) * kKB) % KWB == 0 || st == nst - 1) {
            const int w = st * kKB / KWB;
            bias(w);
            __syncthreads();
            if (w + 1 < nwin) put_win_scales(w + 1);
            load_win_scales(w + 2 < nwin ? w + 2 : nwin - 1);
        }
    };

    // ---- prologue ----
    load_quad(0);
    load_win_scales(0);
    fetch(0);
    put_win_scales(0);
    load_win_scales(nwin > 1 ? 1 : 0);
    commit(0, 0);
    fetch(1);
    __syncthreads();

    // ---- main loop: stages in pairs (one quad of blocks); all global loads
    // unconditional (indices past the end clamped; those copies never used) ----
    for (int st = 0; st < nst; st += 2) {
        const int s2 = st + 2 < nst ? st + 2 : nst - 1;
        const int s3 = st + 3 < nst ? st + 3 : nst - 1;
        swap_quad();
        load_quad(s2 / 2);
        // the next stage's X conversion shares a basic block with this
        // stage's MFMAs; the FMAs complete before the window's branch
        compute(0, st, 0);
        commit(1, st + 1);
        fetch(s2);
        pin();
        window_end(st);
        __syncthreads();
        compute(1, st + 1, 2);
        commit(0, s2);  // past the end: a copy of the last stage, never read
        fetch(s3);
        pin();
        window_end(st + 1);
        __syncthreads();
    }

    // store: lane (h, n) holds tokens 32 tt + 8 (v / 4) + 4 h + v % 4 of weight
    // row 64 wm + 32 rt + n (K splits: added to the zeroed y)
    const bool split_k = sp.ks > 1;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        const int64_t r = row0 + 64 * wm + 32 * rt + n32;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t t = tok0 + 32 * tt + 8 * (v >> 2) + 4 * h + (v & 3);
                if (r < M && t < N) {
                    float* const o = y + t * M + r;
                    if (split_k)
                        unsafeAtomicAdd(o, acc[rt][tt][v]);
                    else
                        *o = acc[rt][tt][v];
                }
            }
    }
}

// y[0 .. n) = 0 (y 16-byte aligned): float4 stores, then the n % 4 tail
__global__ void zero_kernel(float* __restrict__ y, int64_t n) {
    const int64_t n4 = n / 4;
    const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t i = i0; i < n4; i += (int64_t)gridDim.x * blockDim.x)
        reinterpret_cast<float4*>(y)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i0 < n - 4 * n4) y[4 * n4 + i0] = 0.f;
}

}  // namespace

int cu_count_pf() {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
        return 256;
    return v;
}

// Work split of a launch over `tiles` (row tile, token tile) pairs: K splits
// on super-block boundaries, the fewest that keep the compute units (one
// workgroup each) at least 85 % busy over the launch's rounds, else the best
// of them; every split keeps at least four super-blocks.
GemmSplit plan_split(int64_t nrt, int64_t ntt, int64_t K, int64_t cus) {
    GemmSplit sp;
    sp.nrt = nrt;
    sp.ntt = ntt;
    const int nsb = (int)(K / 256);
    const int64_t tiles = nrt * ntt;
    if (cus <= 0) cus = cu_count_pf();
    const int kmax = nsb / 4 > 1 ? nsb / 4 : 1;
    int best = 1;
    double best_eff = 0.0;
    for (int ks = 1; ks <= kmax && ks <= 64; ++ks) {
        const int64_t g = tiles * ks;
        const double eff = (double)g / (double)(((g + cus - 1) / cus) * cus);
        if (eff > best_eff + 1e-9) {
            best = ks;
            best_eff = eff;
        }
        if (eff >= 0.85) break;
    }
    sp.sbp = (nsb + best - 1) / best;
    sp.ks = (nsb + sp.sbp - 1) / sp.sbp;
    return sp;
}

// y = 0 ahead of a K-split launch (its partial results are added atomically)
void zero_fill(float* y, int64_t n, hipStream_t stream) {
    const int64_t zb = (n / 4 + 255) / 256 < 16384 ? (n / 4 + 255) / 256 + 1 : 16384;
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)zb), dim3(256), 0, stream, y, n);
}

namespace {

template <int FMT, int WM, int TT>
hipError_t launch_tile(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                       const Planes& p, hipStream_t stream) {
    using TL = GemmTile<WM, TT>;
    const GemmSplit sp = plan_split((M + TL::BM - 1) / TL::BM, (n_tok + TL::BN - 1) / TL::BN, K);
    const int64_t grid = sp.nrt * sp.ntt * sp.ks;
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (query_only(kernel_name<Name_gemm_kernel, FMT, WM, TT>(), sp.ks > 1 ? 2 : 1)) return hipSuccess;
    if (sp.ks > 1) zero_fill(y, n_tok * M, stream);
    hipLaunchKernelGGL((gemm_kernel<FMT, WM, TT>), dim3((unsigned)grid), dim3(TL::NT),
                       TL::bytes(MF<FMT>::kSums), stream, W, x, y, M, K, n_tok, p.off1, p.off2, sp);
    return hipGetLastError();
}

template <int FMT, int WM>
hipError_t launch_tile32(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                         const Planes& p, hipStream_t stream) {
    using TL = Tile32<WM>;
    const GemmSplit sp = plan_split((M + TL::BM - 1) / TL::BM, (n_tok + TL::BN - 1) / TL::BN, K);
    const int64_t grid = sp.nrt * sp.ntt * sp.ks;
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (query_only(kernel_name<Name_gemm32_kernel, FMT, WM>(), sp.ks > 1 ? 2 : 1)) return hipSuccess;
    if (sp.ks > 1) zero_fill(y, n_tok * M, stream);
    // scale planes in the first two offset slots, the fifth-bit plane apart
    int64_t o1 = p.off1, o2 = p.off2, oh = 0;
    if constexpr (FMT == LW_Q5_0 || FMT == LW_Q5_1 || FMT == LW_Q5_K || FMT == LW_Q6_K) {
        o1 = p.off2;
        o2 = p.off3;
        oh = p.off1;
    }  // Q2_K: its 2-bit code plane is plane 0 (oh = 0), the scales planes 1 and 2
    hipLaunchKernelGGL((gemm32_kernel<FMT, WM>), dim3((unsigned)grid), dim3(TL::NT), TL::bytes(), stream, W, x, y,
                       M, K, n_tok, o1, o2, oh, sp);
    return hipGetLastError();
}

template <int FMT>
hipError_t launch_gemm(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                       const Planes& p, hipStream_t stream) {
    // Q8_0: 16 x 16 tiles (two code words per block and lane in flight), half
    // the token tiles; the 4-bit formats: 32 x 32 tiles
    if constexpr (FMT == LW_Q8_0)
        return launch_tile<FMT, 4, 2>(W, x, y, M, K, n_tok, p, stream);
    else
        return launch_tile32<FMT, 8>(W, x, y, M, K, n_tok, p, stream);
}

}  // namespace

hipError_t launch_prefill(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                          int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_gemm<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_gemm<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_gemm<LW_Q4_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_gemm<LW_Q8_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_0: return launch_gemm<LW_Q5_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_1: return launch_gemm<LW_Q5_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_K: return launch_gemm<LW_Q5_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_MXFP4: return launch_gemm<LW_MXFP4>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q6_K: return launch_gemm<LW_Q6_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q2_K: return launch_gemm<LW_Q2_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q1_0: return launch_gemm<LW_Q1_0>(W, x, y, M, K, n_tok, p, stream);
    default:
        // f16 weights: token blocks of the matrix-vector kernel
        // (float32 throughout), all whole blocks in one launch
        return launch_gemv_blocks(fmt, W, x, y, M, K, n_tok, p, stream);
    }
}

}  // namespace lw
