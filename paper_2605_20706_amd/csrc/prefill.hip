// Prefill product on the matrix cores (n_tok > 16; the 4-bit and 8-bit formats).
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k]. With many tokens the product is
// a contraction over K with a token dimension, so it runs on
// v_mfma_f32_16x16x32_bf16 (Sec. 3.2: matrix multiplication tiles through
// shared memory and uses the cooperative matrix instructions of the device;
// Sec. 3.3: quantized blocks are dequantized on the way in and each decoded
// tile is reused for every token of the workgroup).
//
// Precision. One MFMA K-step is one 32-element block. The weight operand holds
// exact bfloat16 values derived from the integer codes only: for the 4-bit
// formats the biased code 128 + q (bits 0x4300 | q), for Q8_0 the code q. X is
// split into bf16 high and low parts (x = hi + lo to 2^-17 relative), two
// MFMAs per tile and block, float32 accumulation. The block's scale, min and
// bias are applied to its float32 partial P:
//   Q4_0:   y += d * P - 136 * d * S     (128 + q = (q - 8) + 136)
//   Q4_K:   y += d*sc * P - (128*d*sc + dmin*m) * S
//   Q8_0:   y += d * P
// where S = sum over the block of (hi + lo), the very values fed to the
// matrix core, so the bias cancels to float32 rounding. The error relative
// to sum_k |w * x| stays near 1e-5.
//
// Layout of one block in the MFMA operands: lane slice s (lanes 16s..16s+15)
// holds 8 of the block's 32 elements. For the 4-bit formats slice s takes the
// 32-bit word s of the block's 16 code bytes, i.e. elements 4s..4s+3 (low
// nibbles) and 16+4s..16+4s+3 (high nibbles); for Q8_0, elements 8s..8s+7.
// The X operand in LDS uses the same order of k.
#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

// names of the kernel templates, for lw_kernel_name
struct Name_gemm_kernel {
    static constexpr const char* base = "gemm_kernel";
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
        } else {
            load_scale(W, off1, off2, row, K, blk0, r);
        }
    }
    __device__ static void coef8(const uint32_t* r, int e, float* c1, float* c2) {
        if constexpr (FMT == LW_Q4_0) {
            const float d = half_bits_to_float((r[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
            *c1 = d;
            *c2 = -136.0f * d;
        } else {
            coef_raw(r, e, c1, c2);
        }
    }
    __device__ static void coef_raw(const uint32_t* r, int blk, float* c1, float* c2) {
        if constexpr (FMT == LW_Q4_0) {
            const float d = half_bits_to_float(r[0]);
            *c1 = d;
            *c2 = -136.0f * d;
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
struct MF<LW_Q8_0> {
    static constexpr bool kSums = false;
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

// Tiled kernel: a workgroup computes kBM weight rows x kBN tokens with
// 2 * kWM waves, wave (wm, wn) owning rows 64*wm .. +64 and tokens
// kTT*16*wn .. as 4 x kTT tiles of 16 x 16. Roles in D = A . B: A is X (16
// tokens x one 32-element block), B the decoded codes (one block x 16 weight
// rows), so lane l holds D[4*(l/16) + v][l % 16] = (token 4*(l/16) + v, weight
// row l % 16) and one coefficient per row tile and block serves its outputs.
//
// The two parts of a block's contribution are accumulated separately:
// c1 * P, one FMA per output and block right after the block's MFMAs, and
// c2 * S, which is itself a product over blocks, sum_b S[t][b] * c2[r][b]:
// block sums and c2 coefficients are gathered for windows of 16 blocks and
// multiplied on the matrix cores once per window (one v_mfma_f32_16x16x16_bf16
// K-step spans the window, with the same output layout), split three ways
// into bf16 parts (exact to 24 bits each), six partial products accumulated
// straight into the output tile. This halves the
// per-block vector work, which bounds this kernel.
//
// K advances in stages of kKB blocks. Per stage the workgroup converts the X
// slab (kBN tokens x 32*kKB values) to hi/lo bf16 and the c1 coefficients of
// its kBM rows into one of two LDS stage buffers (one barrier per stage), and
// appends block sums and c2 to the window buffer (one barrier more per window). Each
// wave loads the codes of its own 64 rows directly into registers, two stages
// ahead. Consecutive workgroups take consecutive token tiles of the same rows,
// so a weight tile is read from HBM once and reused from L2.
constexpr int kWM = 2, kBM = 64 * kWM, kTT = 2, kBN = 32 * kTT, kKB = 2, kGT = 128 * kWM;
constexpr int kWin = 16;       // blocks per window (coefficients; the c2 * S product: one 16x16x16 MFMA K-step)
constexpr int kWp = kWin + 1;  // padded row of the S / c2 window buffers (bank-conflict free writes)

struct GemmLds {
    static constexpr int kX = kKB * 4 * kBN;                       // bf16x8 entries per half per stage
    static constexpr size_t kStage = (size_t)2 * kX * 16;          // stage buffer: xh, xl [kKB][4][kBN]
    static constexpr size_t kC1 = (size_t)kWin * kBM * 4;          // c1 of a window [kWin][kBM]
    static constexpr size_t kWinB = (size_t)(kBN + kBM) * kWp * 4;  // S [kBN][kWp], c2 [kBM][kWp]
    static constexpr size_t kBytes = 2 * kStage + 2 * kC1 + kWinB;
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

template <int FMT>
__global__ void __launch_bounds__(kGT) __attribute__((amdgpu_waves_per_eu(2, 2)))
    gemm_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                int64_t K, int64_t N, int64_t off1, int64_t off2) {
    using T = MF<FMT>;
    constexpr bool kQ4 = FMT != LW_Q8_0;
    extern __shared__ bf16x8 smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % kWM, wn = wave / kWM;
    const int i16 = lane & 15, s4 = lane >> 4;
    const int64_t ntt = (N + kBN - 1) / kBN;
    const int64_t row0 = (int64_t)(blockIdx.x / ntt) * kBM;
    const int64_t tok0 = (int64_t)(blockIdx.x % ntt) * kBN;
    const uint32_t K32 = (uint32_t)K;
    const int nblk = (int)(K / 32);
    const int nst = nblk / kKB;  // K is a multiple of 256: a multiple of 4 stages
    const int nwin = (nblk + kWin - 1) / kWin;

    char* lds = reinterpret_cast<char*>(smem);
    auto st_xh = [&](int bf) __attribute__((always_inline)) { return reinterpret_cast<bf16x8*>(lds + bf * GemmLds::kStage); };
    auto st_xl = [&](int bf) __attribute__((always_inline)) { return st_xh(bf) + GemmLds::kX; };
    auto win_c1 = [&](int w) __attribute__((always_inline)) {
        return reinterpret_cast<float*>(lds + 2 * GemmLds::kStage + (w & 1) * GemmLds::kC1);
    };
    float* win_s = reinterpret_cast<float*>(lds + 2 * GemmLds::kStage + 2 * GemmLds::kC1);  // [kBN][kWp]
    float* win_c2 = win_s + kBN * kWp;                                                      // [kBM][kWp]

    // ---- codes of this lane's rows (B operand columns), clamped; stores are masked ----
    uint64_t wrow[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int64_t r = row0 + 64 * wm + 16 * rt + i16;
        wrow[rt] = (uint64_t)(r < M ? r : M - 1);
    }
    // 4-bit formats: a quad = 4 blocks = 2 stages; lane (s4, i16) loads block
    // 4q + s4 of its row (16 bytes) and a register transpose hands it word s4
    // of each of the 4 blocks. Q8_0: per stage, word s4 of each block.
    u32x4v qraw[4], qcur[4];
    using Word8 = uint64_t;
    Word8 cwA[4][kKB], cwB[4][kKB];
    auto load_quad = [&](int q) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
            qraw[rt] = *reinterpret_cast<const u32x4v*>(W + wrow[rt] * (K32 / 2u) + 16u * (uint32_t)(4 * q + s4));
    };
    auto load_codes8 = [&](Word8 (*cw)[kKB], int st) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int b = 0; b < kKB; ++b)
                cw[rt][b] = *reinterpret_cast<const uint64_t*>(W + wrow[rt] * K32 + 32u * (uint32_t)(st * kKB + b) + 8u * s4);
    };

    // ---- window coefficients: thread (row cr, half ch) handles blocks 8ch..8ch+7 of a window ----
    static_assert(kGT == 2 * kBM && kWin == 16, "one 8-block scale item per thread");
    const int cr = tid % kBM, ch = tid / kBM;
    const int64_t crow = row0 + cr < M ? row0 + cr : M - 1;
    uint32_t sraw[4];
    auto load_win_scales = [&](int w) __attribute__((always_inline)) {
        int blk0 = w * kWin + 8 * ch;
        blk0 = blk0 < nblk ? blk0 : nblk - 8;  // past the end: a valid copy, never used
        T::load_scale8(W, off1, off2, (uint64_t)crow, K32, blk0, sraw);
    };
    auto put_win_scales = [&](int w) __attribute__((always_inline)) {
        float* c1w = win_c1(w);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float c1, c2;
            T::coef8(sraw, e, &c1, &c2);
            c1w[(8 * ch + e) * kBM + cr] = c1;
            if constexpr (T::kSums) win_c2[cr * kWp + 8 * ch + e] = c2;
        }
    };

    // ---- X stage producer: items (block, token, slice) ----
    constexpr int kXI = kKB * kBN * 4 / kGT;
    float4 xa[kXI], xb[kXI];
    auto fetch = [&](int st) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kXI; ++i) {
            const int it = tid + i * kGT;
            const int sl = it & 3, t = (it >> 2) % kBN, b = (it >> 2) / kBN;
            // tokens past N read the last token: their outputs are never stored
            const int64_t tt = tok0 + t < N ? tok0 + t : N - 1;
            const float* xp = x + tt * K + 32 * (int64_t)(st * kKB + b);
            xa[i] = *reinterpret_cast<const float4*>(xp + T::x_first(sl, 0));
            xb[i] = *reinterpret_cast<const float4*>(xp + T::x_first(sl, 1));
        }
    };
    auto commit = [&](int bf, int st) __attribute__((always_inline)) {
        bf16x8* xh = st_xh(bf);
        bf16x8* xl = st_xl(bf);
#pragma unroll
        for (int i = 0; i < kXI; ++i) {
            const int it = tid + i * kGT;
            const int sl = it & 3, t = (it >> 2) % kBN, b = (it >> 2) / kBN;
            const float v[8] = {xa[i].x, xa[i].y, xa[i].z, xa[i].w, xb[i].x, xb[i].y, xb[i].z, xb[i].w};
            bf16x8 h, l;
            float sum = split_bf16x8(v, &h, &l);
            // token slots are XOR-swizzled by the slice so that the four
            // slices written by a lane quad fall into different LDS banks
            xh[(b * 4 + sl) * kBN + (t ^ (sl << 2))] = h;
            xl[(b * 4 + sl) * kBN + (t ^ (sl << 2))] = l;
            if constexpr (T::kSums) {
                const int blk = st * kKB + b;
                sum += dpp_move<0xB1>(sum);  // the 4 slices of (block, token) are one lane quad
                sum += dpp_move<0x4E>(sum);
                if (sl == 0) win_s[t * kWp + blk % kWin] = sum;
            }
        }
    };

    f32x4 acc[4][kTT];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int tt = 0; tt < kTT; ++tt) acc[rt][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // stage st from LDS buffer bf; the codes of its block b: word j0 + b of
    // qcur (4-bit) or cw[.][b] (Q8_0)
    auto compute = [&](int bf, int st, int j0, Word8 (*cw)[kKB]) __attribute__((always_inline)) {
        const bf16x8* xh = st_xh(bf);
        const bf16x8* xl = st_xl(bf);
#pragma unroll
        for (int b = 0; b < kKB; ++b) {
            const int blk = st * kKB + b;
            const float* c1s = win_c1(blk / kWin) + (blk % kWin) * kBM;
            bf16x8 ah[kTT], al[kTT];
#pragma unroll
            for (int tt = 0; tt < kTT; ++tt) {
                const int t = (16 * kTT * wn + 16 * tt + i16) ^ (s4 << 2);
                ah[tt] = xh[(b * 4 + s4) * kBN + t];
                al[tt] = xl[(b * 4 + s4) * kBN + t];
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                bf16x8 bw;
                if constexpr (kQ4)
                    bw = T::decode(qcur[rt][j0 + b]);
                else
                    bw = T::decode(cw[rt][b]);
                const float c1 = c1s[64 * wm + 16 * rt + i16];
#pragma unroll
                for (int tt = 0; tt < kTT; ++tt) {
                    f32x4 p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[tt], bw, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[tt], bw, p, 0, 0, 0);
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[rt][tt][v] = __builtin_fmaf(c1, p[v], acc[rt][tt][v]);
                }
            }
        }
    };
    // acc += S(window) . c2(window)^T for window w (nv valid blocks; the rest masked)
    auto bias = [&](int w) __attribute__((always_inline)) {
        const int nv = nblk - w * kWin < kWin ? nblk - w * kWin : kWin;
        bf16x4 sh[kTT], sm[kTT], sl[kTT];
#pragma unroll
        for (int tt = 0; tt < kTT; ++tt) {
            const float* sp = win_s + (16 * kTT * wn + 16 * tt + i16) * kWp + 4 * s4;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = 4 * s4 + e < nv ? sp[e] : 0.f;
            split3_bf16x4(v, &sh[tt], &sm[tt], &sl[tt]);
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            const float* cp = win_c2 + (64 * wm + 16 * rt + i16) * kWp + 4 * s4;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = 4 * s4 + e < nv ? cp[e] : 0.f;
            bf16x4 chh, chm, chl;
            split3_bf16x4(v, &chh, &chm, &chl);
#pragma unroll
            for (int tt = 0; tt < kTT; ++tt) {
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
    // after stage st: when it ends a window, the window's c2 * S product is
    // added, and (after a barrier: the window buffers are reused) the next
    // window's coefficients are stored and the one after is prefetched
    auto window_end = [&](int st) __attribute__((always_inline)) {
        if (((st + 1) * kKB) % kWin == 0 || st == nst - 1) {
            const int w = st * kKB / kWin;
            if constexpr (T::kSums) bias(w);
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
        compute(0, st, 0, cwA);
        window_end(st);
        if constexpr (!kQ4) load_codes8(cwA, s2);
        commit(1, st + 1);
        fetch(s2);
        __syncthreads();
        compute(1, st + 1, 2, cwB);
        window_end(st + 1);
        if constexpr (!kQ4) load_codes8(cwB, s3);
        commit(0, s2);  // past the end: a copy of the last stage, never read
        fetch(s3);
        __syncthreads();
    }

    // store: lane holds tokens 16*kTT*wn + 16*tt + 4*s4 + v of weight row 64*wm + 16*rt + i16
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int64_t r = row0 + 64 * wm + 16 * rt + i16;
        if (r >= M) continue;
#pragma unroll
        for (int tt = 0; tt < kTT; ++tt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t t = tok0 + 16 * kTT * wn + 16 * tt + 4 * s4 + v;
                if (t < N) y[t * M + r] = acc[rt][tt][v];
            }
    }
}

template <int FMT>
hipError_t launch_gemm(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                       const Planes& p, hipStream_t stream) {
    const int64_t grid = ((M + kBM - 1) / kBM) * ((n_tok + kBN - 1) / kBN);
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (query_only(kernel_name<Name_gemm_kernel, FMT>())) return hipSuccess;
    hipLaunchKernelGGL((gemm_kernel<FMT>), dim3((unsigned)grid), dim3(kGT), GemmLds::kBytes, stream, W, x, y, M, K,
                       n_tok, p.off1, p.off2);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                          int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_gemm<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_gemm<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_gemm<LW_Q8_0>(W, x, y, M, K, n_tok, p, stream);
    default:
        // f16 weights: token blocks of the matrix-vector kernel (float32 throughout)
        for (int64_t t0 = 0; t0 < n_tok; t0 += LW_GEMV_MAX_TOK) {
            const int64_t nt = (n_tok - t0) < LW_GEMV_MAX_TOK ? (n_tok - t0) : LW_GEMV_MAX_TOK;
            const hipError_t err = launch_gemv(fmt, W, x + t0 * K, y + t0 * M, M, K, nt, p, stream);
            if (err != hipSuccess) return err;
        }
        return hipSuccess;
    }
}

}  // namespace lw
