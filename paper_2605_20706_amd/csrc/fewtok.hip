// Few-token product (2 <= n_tok <= 8) on the matrix cores for every quantized
// format but Q8_0, with the activations converted once per workgroup.
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k]: the decode product of Sec. 2.1
// for a small batch of tokens. The weights are read from HBM exactly once and
// dequantized in registers (Sec. 3.3); the contraction runs on
// v_mfma_f32_16x16x32_bf16, one MFMA K step per 32-element block, so each
// block's scale applies to its own partial product.
//
// MFMA roles (layout in lw_mfma.hpp): A = the activations, 16 rows = the bf16
// high parts of tokens 0..7 (rows 0..7) and the bf16 low parts (rows 8..15);
// B = the biased codes 128 + q of 16 weight rows; D[4g+v][n] = token half
// 4g+v of weight row n. Rows of tokens >= n_tok are zero.
//
// Work split: workgroup b owns the rows [b*rpw, min((b+1)*rpw, M)), about
// M / #CU of them, so every compute unit streams the same number of weight
// bytes. They form ntq tiles of 16 rows (a tile past the last row repeats
// it). The nw waves are nw/P tile slots x P parts of K: wave w serves tiles
// w/P, w/P + nw/P, ... and, of every window of ws super-blocks (256 columns
// each), the (w mod P)-th of P equal parts. The unit of work is one
// super-block of one tile: 16 rows x 128 code bytes (two 16-byte loads per
// lane: lane (g, n) loads block 4h + g of row n, and a transpose across the
// lane groups gives it word g of blocks 4h..4h+3) plus the super-block's
// scales. Each wave keeps two units in flight; the loads of a unit are issued
// two units ahead of its use, across window boundaries.
//
// Activations: per window, all threads convert X[t][window] into LDS in the
// A layout (8 KiB per super-block): thread item (t, block, g) reads the two
// float4 of its lane group's elements, splits them into bf16 high and low
// parts and writes one 16-byte slot of row t and one of row 8 + t. The MFMA
// reads one slot per lane per block. Barriers wait only for LDS, never for the
// weight loads in flight.
//
// Precision (the reading shared by the matrix-core paths): the codes enter as
// the exact bf16 of 128 + q (the 5-bit formats: the fifth bit merged into q
// first); X = high + low to 16 significant bits; per block
// y += c1 * (P + k * S) + dm * (k * S)-term, with S the block sum of the
// multiplied operand, computed by the same MFMA against a B of the constant k
// and used as P's accumulator:
//   Q4_0:     w = d (q - 8)         -> c1 = d,    k = -136, dm = 0
//   Q5_0:     w = d (q - 16)        -> c1 = d,    k = -144, dm = 0
//   Q4_K, Q5_K: w = d sc q - dmin m -> c1 = d sc, k = -128, dm = dmin m / 128
//   Q4_1, Q5_1: w = d q + m         -> c1 = d,    k = -128, dm = -m / 128
// MXFP4 multiplies the exact bf16 of its e2m1 values (no offset, no k * S):
// y += 2^(E - 127) * P. Q6_K and Q2_K scale 16-element sub-blocks: a block
// is two v_mfma_f32_16x16x16_bf16 (the low and the high half of each lane's
// 8 operand values, elements 0..15 and 16..31 of the block), each with its
// own coefficients (q1_0: the bf16 +-1 of each bit, y += d * P):
//   Q6_K:     w = d sc (q - 32)     -> c1 = d sc, k = -160, dm = 0
//   Q2_K:     w = d sc q - dmin m   -> c1 = d sc, k = -128, dm = dmin m / 128
// Accumulation is f32 throughout.
#include "lw_internal.hpp"
#include "lw_mfma.hpp"

namespace lw {
namespace {

struct Name_fewtok_kernel {
    static constexpr const char* base = "fewtok_kernel";
};

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kFtMaxWaves = 16;  // waves per workgroup
constexpr int kFtWinSB = 16;     // super-blocks per window: 16 x 8 blocks x 1 KiB of A = 128 KiB of LDS
constexpr int kFtMaxTpw = 4;     // tiles per wave when the waves do not split K
template <int FMT>
constexpr int kFtRing = FMT == LW_Q4_0 ? 3 : 2;  // units in flight per wave (fewer where the scales take more registers)
template <int FMT>
constexpr bool kFtQ5 = FMT == LW_Q5_0 || FMT == LW_Q5_1 || FMT == LW_Q5_K;
template <int FMT>
constexpr bool kFtSub16 = FMT == LW_Q6_K || FMT == LW_Q2_K;

// Scale data of one super-block (8 blocks, 256 columns) of one weight row.
template <int FMT>
struct SbScale;

template <>
struct SbScale<LW_Q4_0> {
    u32x4 d;  // binary16 d of the 8 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t sbi) {
        d = *reinterpret_cast<const u32x4*>(P1 + 16 * sbi);
    }
    // c1 of blocks 4h .. 4h+3 (d); dm is unused
    __device__ void coef(int h, float* c1, float*) const {
        const uint32_t a = h ? d[2] : d[0], b = h ? d[3] : d[1];
        c1[0] = half_bits_to_float(a & 0xFFFFu);
        c1[1] = half_bits_to_float(a >> 16);
        c1[2] = half_bits_to_float(b & 0xFFFFu);
        c1[3] = half_bits_to_float(b >> 16);
    }
};

template <>
struct SbScale<LW_Q4_1> {
    u32x4 dm[2];  // {binary16 d, binary16 m} of the 8 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t sbi) {
        dm[0] = *reinterpret_cast<const u32x4*>(P1 + 32 * sbi);
        dm[1] = *reinterpret_cast<const u32x4*>(P1 + 32 * sbi + 16);
    }
    // c1 = d and dm = -m / 128 of blocks 4h .. 4h+3
    __device__ void coef(int h, float* c1, float* dmo) const {
        const u32x4 v = h ? dm[1] : dm[0];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            c1[i] = half_bits_to_float(v[i] & 0xFFFFu);
            dmo[i] = half_bits_to_float(v[i] >> 16) * (-1.0f / 128.0f);
        }
    }
};

template <>
struct SbScale<LW_Q4_K> {
    uint32_t r0, r1, r2, dd;  // the 96-bit scale record and {d, dmin}
    __device__ void load(const uint8_t* P1, const uint8_t* P2, uint64_t sbi) {
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(P1 + 12 * sbi);
        r0 = rec[0];
        r1 = rec[1];
        r2 = rec[2];
        dd = *reinterpret_cast<const uint32_t*>(P2 + 4 * sbi);
    }
    // c1 = d * sc_j and dm = dmin * m_j / 128 of sub-blocks j = 4h .. 4h+3:
    // sc_j sits at record bit 6j, m_j at bit 48 + 6j (one funnel shift each;
    // h is a compile-time constant at every use, so the word choice is too)
    __device__ void coef(int h, float* c1, float* dm) const {
        const float d = half_bits_to_float(dd & 0xFFFFu), dmin = half_bits_to_float(dd >> 16) * (1.0f / 128.0f);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t j = 4u * (uint32_t)h + (uint32_t)i;
            const uint32_t ts = 6u * j, tm = 16u + 6u * j;
            const uint32_t sc_w = __builtin_amdgcn_alignbit(r1, ts < 32u ? r0 : r1, ts & 31u);
            const uint32_t m_w = __builtin_amdgcn_alignbit(r2, tm < 32u ? r1 : r2, tm & 31u);
            c1[i] = d * (float)(sc_w & 63u);
            dm[i] = dmin * (float)(m_w & 63u);
        }
    }
};

// The 5-bit formats read Q4_0's, Q4_1's and Q4_K's scale data from their own
// planes (the kernel passes those planes).
template <>
struct SbScale<LW_Q5_0> : SbScale<LW_Q4_0> {};
template <>
struct SbScale<LW_Q5_1> : SbScale<LW_Q4_1> {};
template <>
struct SbScale<LW_Q5_K> : SbScale<LW_Q4_K> {};

template <>
struct SbScale<LW_Q1_0> {
    uint32_t d2;  // the binary16 d of the super-block's two 128-element groups
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t sbi) {
        d2 = *reinterpret_cast<const uint32_t*>(P1 + 4 * sbi);
    }
    // c1 = d of blocks 4h .. 4h+3 (all in group h); dm is unused
    __device__ void coef(int h, float* c1, float*) const {
        const float d = half_bits_to_float(h ? d2 >> 16 : d2 & 0xFFFFu);
#pragma unroll
        for (int i = 0; i < 4; ++i) c1[i] = d;
    }
};

template <>
struct SbScale<LW_MXFP4> {
    uint32_t e[2];  // the e8m0 exponent bytes of the 8 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t sbi) {
        const uint2 v = *reinterpret_cast<const uint2*>(P1 + 8 * sbi);
        e[0] = v.x;
        e[1] = v.y;
    }
    // c1 = 2^(E - 127) of blocks 4h .. 4h+3; dm is unused
    __device__ void coef(int h, float* c1, float*) const {
        const uint32_t w = h ? e[1] : e[0];
#pragma unroll
        for (int i = 0; i < 4; ++i) c1[i] = e8m0_to_float((w >> (8 * i)) & 0xFFu);
    }
};

// 16-element sub-blocks: the 16 coefficient units of a super-block, read at
// once (16 bytes of scales, then d or {d, dmin}).
template <>
struct SbScale<LW_Q6_K> {
    u32x4 sc;     // signed 8-bit sub-block scales
    uint32_t d;   // binary16 d
    __device__ void load(const uint8_t* P1, const uint8_t* P2, uint64_t sbi) {
        sc = *reinterpret_cast<const u32x4*>(P1 + 16 * sbi);
        d = *reinterpret_cast<const uint16_t*>(P2 + 2 * sbi);
    }
    // c1 = d * sc of sub-blocks 8h .. 8h+7; dm is unused
    __device__ void coef16(int h, float* c1, float*) const {
        const float dv = half_bits_to_float(d);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t w = sc[2 * h + (i >> 2)];
            c1[i] = dv * (float)(int)(int8_t)(uint8_t)(w >> (8 * (i & 3)));
        }
    }
};
template <>
struct SbScale<LW_Q2_K> {
    u32x4 scm;    // {scale, min} nibbles of the sub-blocks
    uint32_t dd;  // {binary16 d, binary16 dmin}
    __device__ void load(const uint8_t* P1, const uint8_t* P2, uint64_t sbi) {
        scm = *reinterpret_cast<const u32x4*>(P1 + 16 * sbi);
        dd = *reinterpret_cast<const uint32_t*>(P2 + 4 * sbi);
    }
    // c1 = d * sc and dm = dmin * m / 128 of sub-blocks 8h .. 8h+7
    __device__ void coef16(int h, float* c1, float* dm) const {
        const float dv = half_bits_to_float(dd & 0xFFFFu), mv = half_bits_to_float(dd >> 16) * (1.0f / 128.0f);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t b = (scm[2 * h + (i >> 2)] >> (8 * (i & 3))) & 0xFFu;
            c1[i] = dv * (float)(b & 15u);
            dm[i] = mv * (float)(b >> 4);
        }
    }
};

template <int FMT>
struct Unit {
    u32x4 c[2];   // code lines: block 8s + 4h + g of the lane's row, h = 0, 1
    u32x4 qh[2];  // the 5-bit formats: fifth bits of blocks 8s + 4h .. 8s + 4h + 3 (one word each)
    u32x4 two;    // Q6_K high bits, Q2_K codes: blocks 8s + 2g, 8s + 2g + 1 (8 bytes each)
    SbScale<FMT> sc;
    int i, s;  // tile (of the wave), super-block
};

// Code word w of a block (lane group g: elements 4g .. 4g+3 in the low
// nibbles, 16 + 4g .. 16 + 4g + 3 in the high ones) with its fifth bits from
// the block's bit word qw (bit e for element e) -> the 8 bf16 values 128 + q.
__device__ __forceinline__ bf16x8 biased_codes5(uint32_t w, uint32_t qw, uint32_t g4) {
    const uint32_t lo = opaque((w & 0x0F0F0F0Fu) | spread4((qw >> g4) << 4 & 0xF0u));
    const uint32_t hi = opaque(((w >> 4) & 0x0F0F0F0Fu) | spread4((qw >> (16u + g4)) << 4 & 0xF0u));
    const uint32_t k43 = 0x43434343u;
    const u32x4 v = {__builtin_amdgcn_perm(k43, lo, 0x04010400u), __builtin_amdgcn_perm(k43, lo, 0x04030402u),
                     __builtin_amdgcn_perm(k43, hi, 0x04010400u), __builtin_amdgcn_perm(k43, hi, 0x04030402u)};
    return __builtin_bit_cast(bf16x8, v);
}

// Q6_K: code word w and the 16 bits hw of the two high bits of its elements
// (bits 0-7: elements 4g .. 4g+3; bits 8-15: 16 + 4g .. 16 + 4g + 3) -> the
// 8 bf16 values 128 + q. Q2_K: the 2-bit codes alone.
__device__ __forceinline__ bf16x8 biased_codes6(uint32_t w, uint32_t hw) {
    const uint32_t lo = opaque((w & 0x0F0F0F0Fu) | spread2_hi(hw & 0xFFu));
    const uint32_t hi = opaque(((w >> 4) & 0x0F0F0F0Fu) | spread2_hi((hw >> 8) & 0xFFu));
    const uint32_t k43 = 0x43434343u;
    const u32x4 v = {__builtin_amdgcn_perm(k43, lo, 0x04010400u), __builtin_amdgcn_perm(k43, lo, 0x04030402u),
                     __builtin_amdgcn_perm(k43, hi, 0x04010400u), __builtin_amdgcn_perm(k43, hi, 0x04030402u)};
    return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ bf16x8 biased_codes2(uint32_t hw) {
    const uint32_t lo = opaque(spread2_lo(hw & 0xFFu));
    const uint32_t hi = opaque(spread2_lo((hw >> 8) & 0xFFu));
    const uint32_t k43 = 0x43434343u;
    const u32x4 v = {__builtin_amdgcn_perm(k43, lo, 0x04010400u), __builtin_amdgcn_perm(k43, lo, 0x04030402u),
                     __builtin_amdgcn_perm(k43, hi, 0x04010400u), __builtin_amdgcn_perm(k43, hi, 0x04030402u)};
    return __builtin_bit_cast(bf16x8, v);
}

// The 2-bit plane of a super-block (lane group L holds the 8-byte records
// of blocks 2L, 2L + 1 as words s0..s3) -> for lane group g the word R_L,
// L = 0..3, holding byte g of each of s0..s3 of lane group L: bytes 0, 1 are
// the two bytes of block 2L its elements need, bytes 2, 3 those of block
// 2L + 1. A byte transpose within the lane (P_d = byte d of s0..s3), then the
// word transpose across the lane groups.
__device__ __forceinline__ u32x4 two_bit_transpose(u32x4 s) {
    const uint32_t t01l = __builtin_amdgcn_perm(s[1], s[0], 0x05010400u);  // s0[0] s1[0] s0[1] s1[1]
    const uint32_t t01h = __builtin_amdgcn_perm(s[1], s[0], 0x07030602u);  // s0[2] s1[2] s0[3] s1[3]
    const uint32_t t23l = __builtin_amdgcn_perm(s[3], s[2], 0x05010400u);
    const uint32_t t23h = __builtin_amdgcn_perm(s[3], s[2], 0x07030602u);
    const u32x4 p = {__builtin_amdgcn_perm(t23l, t01l, 0x05040100u), __builtin_amdgcn_perm(t23l, t01l, 0x07060302u),
                     __builtin_amdgcn_perm(t23h, t01h, 0x05040100u), __builtin_amdgcn_perm(t23h, t01h, 0x07060302u)};
    return quad_transpose(p);
}

// q1_0: the block's code bits qw (bit e for element e) -> the bf16 +-1 of
// the lane group's 8 elements, in the order above.
__device__ __forceinline__ bf16x8 sign_codes(uint32_t qw, uint32_t g4) {
    uint32_t p[4];
    sign_pairs((qw >> g4) & 15u, &p[0], &p[1]);
    sign_pairs((qw >> (16u + g4)) & 15u, &p[2], &p[3]);
    return __builtin_bit_cast(bf16x8, (u32x4{p[0], p[1], p[2], p[3]}));
}

// Code word w of an MXFP4 block -> the bf16 values of its 8 e2m1 codes, in
// the same element order.
__device__ __forceinline__ bf16x8 fp4_codes(uint32_t w) {
    uint32_t p[4];
    fp4_pairs(opaque(w & 0x07070707u), (w << 4) & 0x80808080u, &p[0], &p[1]);
    fp4_pairs(opaque((w >> 4) & 0x07070707u), w & 0x80808080u, &p[2], &p[3]);
    return __builtin_bit_cast(bf16x8, (u32x4{p[0], p[1], p[2], p[3]}));
}

// LDS-only barrier: waits for this wave's LDS traffic, not for its global
// loads (the weight units in flight stay in flight).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int FMT, int TPW, int NS>
__global__ void __launch_bounds__(64 * kFtMaxWaves)
    fewtok_kernel(const RowSegs<NS> sg, const float* __restrict__ x, int K, int ntok, int rpw, int ntq, int P,
                  int ws) {
    extern __shared__ uint4 lds[];
    // the workgroup's matrix (lw_matvec_multi: segment si holds workgroups
    // wg0[si] ..; a workgroup never spans two matrices)
    int si = 0;
#pragma unroll
    for (int k = 1; k < NS; ++k)
        if ((int64_t)blockIdx.x >= sg.wg0[k]) si = k;
    const uint8_t* const W = sg.W[si];
    float* const y = sg.y[si];
    const int M = (int)sg.M[si];
    const int64_t wgi = (int64_t)blockIdx.x - sg.wg0[si];
    const int nthr = blockDim.x;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, n = lane & 15;
    const int nslots = (nthr >> 6) / P;
    const int ts = wave / P, kp = wave - ts * P;
    const int nsb = K >> 8;
    const int nwin = (nsb + ws - 1) / ws;
    const int64_t r0 = wgi * rpw;
    const int64_t rl = (r0 + rpw < (int64_t)M ? r0 + rpw : (int64_t)M) - 1;  // last row of the workgroup
    // scale planes (the 5-bit formats: planes 2 and 3; plane 1 holds the fifth bits)
    // (Q6_K: plane 1 holds the high bits, planes 2 and 3 the scales; Q2_K:
    // plane 0 holds its 2-bit codes, planes 1 and 2 the scales)
    constexpr bool kQ5 = kFtQ5<FMT>;
    constexpr bool kFp4 = FMT == LW_MXFP4;
    constexpr bool kSub16 = kFtSub16<FMT>;
    constexpr bool kQ2 = FMT == LW_Q2_K;
    constexpr bool kQ1 = FMT == LW_Q1_0;  // its code bits are read as the fifth-bit words
    const bool hi_planes = kQ5 || FMT == LW_Q6_K;
    const uint8_t* PH = W + (kQ2 || kQ1 ? 0 : sg.off1[si]);
    const uint8_t* P1 = W + (hi_planes ? sg.off2[si] : sg.off1[si]);
    const uint8_t* P2 = W + (hi_planes ? sg.off3[si] : sg.off2[si]);
    const uint64_t rowb = (uint64_t)K / 2u;  // code bytes per row

    // the wave's tiles: the lane's row in each (past the workgroup's last row:
    // that row again, whose lines are read anyway)
    int ntl = 0;
#pragma unroll
    for (int i = 0; i < TPW; ++i)
        if (ts + i * nslots < ntq) ntl = i + 1;
    auto row_of = [&](int i) __attribute__((always_inline)) {
        const int64_t rr = r0 + 16 * (int64_t)(ts + i * nslots) + n;
        return (uint64_t)(rr <= rl ? rr : rl);
    };

    // The wave's units of window w: for each of its ntl tiles, the
    // super-blocks [w*ws + kp*cnt/P, w*ws + (kp+1)*cnt/P), cnt = the
    // window's super-blocks; unit u of the window is tile u / len,
    // super-block a + u mod len. All wave-uniform scalar work.
    auto part = [&](int win, int& a, int& len) __attribute__((always_inline)) {
        const int w0 = win * ws;
        const int cnt = (nsb - w0) < ws ? (nsb - w0) : ws;
        a = w0 + (kp * cnt) / P;
        len = w0 + ((kp + 1) * cnt) / P - a;
    };
    int wa = 0, wlen = 0, wn = 0;  // the current window's part and unit count
    // Loads unit u of the current window into stage st; past the window's
    // last unit (or with no unit at all) it loads that last unit (or the
    // window's first super-block of the first tile) again, so every load is
    // issued unconditionally.
    auto load = [&](Unit<FMT>& st, int u) __attribute__((always_inline)) {
        int i = 0, sb = wa < nsb ? wa : nsb - 1;
        if (wn > 0) {
            const int ue = u < wn ? u : wn - 1;
            i = ue / wlen;
            sb = wa + (ue - i * wlen);
        }
        const uint64_t r = row_of(i);
        if constexpr (!kQ2 && !kQ1) {
            const uint8_t* cp = W + r * rowb + 128u * (uint32_t)sb + 16u * (uint32_t)g;
            st.c[0] = *reinterpret_cast<const u32x4*>(cp);
            st.c[1] = *reinterpret_cast<const u32x4*>(cp + 64);
        }
        if constexpr (kSub16)
            st.two = *reinterpret_cast<const u32x4*>(PH + r * ((uint64_t)K / 4u) + 64u * (uint32_t)sb + 16u * (uint32_t)g);
        if constexpr (kQ5 || kQ1) {
            const uint8_t* hq = PH + r * ((uint64_t)K / 8u) + 32u * (uint32_t)sb;
            st.qh[0] = *reinterpret_cast<const u32x4*>(hq);
            st.qh[1] = *reinterpret_cast<const u32x4*>(hq + 16);
        }
        st.sc.load(P1, P2, r * (uint64_t)nsb + (uint64_t)sb);
        st.i = i;
        st.s = sb;
    };

    // X window -> LDS in the A layout. Slot of (window block lb, lane group
    // gg, A row a): lb*64 + gg*16 + ((a + 4*gg) & 15). The MFMA read of a
    // block (lane (g, n) reads row n of lane group g) covers 64 distinct
    // slots, and consecutive conversion items write distinct 16-byte bank
    // groups. An item is (window block lb, token t < n_tok, lane group gg),
    // item index = 4 (lb * n_tok + t) + gg: two float4 loads, a high/low split
    // and two 16-byte writes (rows t and 8 + t). Rows of absent tokens are
    // zeroed in the first window and stay zero. A batch issues the loads of
    // kXb items per thread before it converts any. The division by n_tok
    // (<= 8) is a multiplication by ceil(2^20 / n_tok), exact for the item
    // counts here (below 2^13 per window).
    constexpr int kXb = (TPW >= 4 || kQ5) ? 2 : 4;  // the 5-bit formats hold more per unit
    const uint32_t tmag = ((1u << 20) + (uint32_t)ntok - 1u) / (uint32_t)ntok;
    auto win_items = [&](int win) __attribute__((always_inline)) {
        const int w0 = win * ws;
        return 32 * ntok * ((nsb - w0) < ws ? (nsb - w0) : ws);  // 4 items per block and token, 8 blocks per super-block
    };
    auto xload = [&](int win, int base, float4* v0, float4* v1) __attribute__((always_inline)) {
        const int items = win_items(win);
#pragma unroll
        for (int k = 0; k < kXb; ++k) {
            // clamped index: every load is issued
            int it = base + tid + k * nthr;
            it = it < items ? it : items - 1;
            const uint32_t q = (uint32_t)it >> 2;
            const int lb = (int)((q * tmag) >> 20);
            const int t = (int)q - lb * ntok;
            const float* xp = x + (int64_t)t * K + 32 * (int64_t)(8 * win * ws + lb) + 4 * (it & 3);
            v0[k] = *reinterpret_cast<const float4*>(xp);
            v1[k] = *reinterpret_cast<const float4*>(xp + 16);
        }
    };
    auto xstore = [&](int win, int base, const float4* v0, const float4* v1) __attribute__((always_inline)) {
        const int items = win_items(win);
#pragma unroll
        for (int k = 0; k < kXb; ++k) {
            const int it = base + tid + k * nthr;
            if (it < items) {
                const int gg = it & 3;
                const uint32_t q = (uint32_t)it >> 2;
                const int lb = (int)((q * tmag) >> 20);
                const int t = (int)q - lb * ntok;
                uint4 hi, lo;
                split_bf16x2(v0[k].x, v0[k].y, hi.x, lo.x);
                split_bf16x2(v0[k].z, v0[k].w, hi.y, lo.y);
                split_bf16x2(v1[k].x, v1[k].y, hi.z, lo.z);
                split_bf16x2(v1[k].z, v1[k].w, hi.w, lo.w);
                lds[lb * 64 + gg * 16 + ((t + 4 * gg) & 15)] = hi;
                lds[lb * 64 + gg * 16 + ((t + 8 + 4 * gg) & 15)] = lo;
            }
        }
    };
    auto convert_rest = [&](int win, int first) __attribute__((always_inline)) {
        const int items = win_items(win);
        for (int base = first; base < items; base += kXb * nthr) {
            float4 w0[kXb], w1[kXb];
            xload(win, base, w0, w1);
            xstore(win, base, w0, w1);
        }
    };
    auto zero_rows = [&]() __attribute__((always_inline)) {
        const int nz = 8 - ntok;
        const int items = 32 * 8 * (nsb < ws ? nsb : ws);  // (block, row slot r < 8, lane group) of window 0
        const uint4 z = {0u, 0u, 0u, 0u};
        for (int it = tid; it < items; it += nthr) {
            const int gg = it & 3;
            const int q = it >> 2;
            const int lb = q >> 3, r = q & 7;  // r < 8: row index among the 8 - ntok absent ones when r < nz
            if (r < nz) {
                const int t = ntok + r;
                lds[lb * 64 + gg * 16 + ((t + 4 * gg) & 15)] = z;
                lds[lb * 64 + gg * 16 + ((t + 8 + 4 * gg) & 15)] = z;
            }
        }
    };

    // bf16 k: -136 (Q4_0: code bias 128 plus the format's offset 8), -144
    // (Q5_0: offset 16) or -128
    // (Q6_K: offset 32, -160)
    const uint32_t kb = FMT == LW_Q4_0   ? 0xC308C308u
                        : FMT == LW_Q5_0 ? 0xC310C310u
                        : FMT == LW_Q6_K ? 0xC320C320u
                                         : 0xC300C300u;
    const bf16x4 bias_b4 = __builtin_bit_cast(bf16x4, (u32x2{kb, kb}));
    const uint32_t g4 = 4u * (uint32_t)g;  // the lane group's first bit in a fifth-bit word
    const bf16x8 bias_b = __builtin_bit_cast(bf16x8, u32x4{kb, kb, kb, kb});
    // the lane's A slot within a block: g * 16 + ((n + 4g) & 15)
    const int aoff = g * 16 + ((n + 4 * g) & 15);

    f32x4 acc[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    int cur = 0;  // the window in LDS
    auto consume = [&](const Unit<FMT>& u) __attribute__((always_inline)) {
        const int b0 = 8 * (u.s - cur * ws);  // window block of the super-block's first block
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if constexpr (kSub16) {
            const u32x4 R = two_bit_transpose(u.two);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                // four blocks, each two sub-blocks: K-steps of 16 over the low
                // and the high half of the lane's operand values
                u32x4 wq = {0u, 0u, 0u, 0u};
                if constexpr (!kQ2) wq = quad_transpose(u.c[h]);
                float c1[8], dm[8];
                u.sc.coef16(h, c1, dm);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int jb = 4 * h + j;
                    const uint32_t hw = (R[jb >> 1] >> (16 * (jb & 1))) & 0xFFFFu;
                    const u32x4 av = __builtin_bit_cast(u32x4, lds[(b0 + jb) * 64 + aoff]);
                    const u32x4 cv = __builtin_bit_cast(u32x4, kQ2 ? biased_codes2(hw) : biased_codes6(wq[j], hw));
#pragma unroll
                    for (int sh = 0; sh < 2; ++sh) {
                        const bf16x4 a4 = __builtin_bit_cast(bf16x4, (u32x2{av[2 * sh], av[2 * sh + 1]}));
                        const bf16x4 c4 = __builtin_bit_cast(bf16x4, (u32x2{cv[2 * sh], cv[2 * sh + 1]}));
                        const f32x4 Cs =
                            __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a4, bias_b4, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                        const f32x4 Ps = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a4, c4, Cs, 0, 0, 0);
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            float o = __builtin_fmaf(c1[2 * j + sh], Ps[v], t[v]);
                            if constexpr (kQ2) o = __builtin_fmaf(dm[2 * j + sh], Cs[v], o);
                            t[v] = o;
                        }
                    }
                }
            }
        } else
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            // four blocks: A slices from LDS, the bias term k * S as an MFMA
            // of A against the constant k, codes decoded, the products with
            // the bias term as accumulator, then the scales
            bf16x8 a[4];
            f32x4 C[4], Pm[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) a[j] = __builtin_bit_cast(bf16x8, lds[(b0 + 4 * h + j) * 64 + aoff]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                C[j] = kFp4 || kQ1 ? f32x4{0.f, 0.f, 0.f, 0.f}
                            : __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], bias_b, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            u32x4 wq = {0u, 0u, 0u, 0u};
            if constexpr (!kQ1) wq = quad_transpose(u.c[h]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                bf16x8 cb;
                if constexpr (kQ1)
                    cb = sign_codes(u.qh[h][j], g4);
                else if constexpr (kQ5)
                    cb = biased_codes5(wq[j], u.qh[h][j], g4);
                else if constexpr (kFp4)
                    cb = fp4_codes(wq[j]);
                else
                    cb = biased_codes(wq[j]);
                Pm[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], cb, C[j], 0, 0, 0);
            }
            float c1[4], dm[4];
            u.sc.coef(h, c1, dm);
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float o = __builtin_fmaf(c1[j], Pm[j][v], t[v]);
                    if constexpr (FMT != LW_Q4_0 && FMT != LW_Q5_0 && !kFp4 && !kQ1)
                        o = __builtin_fmaf(dm[j], C[j][v], o);
                    t[v] = o;
                }
        }
        // add to the unit's tile without a branch (a branch here costs the
        // loop its exact load waits)
        if constexpr (TPW == 1) {
            acc[0] += t;
        } else {
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
                const f32x4 z = {0.f, 0.f, 0.f, 0.f};
                acc[i] += u.i == i ? t : z;
            }
        }
    };

    // Per window: the first x batch's loads, then the window's first kFtRing
    // units' weight loads (both issued while the previous window is still in
    // use), then, once every wave is done with the previous window, the
    // conversion; the weights stream in meanwhile. Within a window the units
    // are consumed in groups of kFtRing, each stage refilled with the unit
    // kFtRing ahead (unconditionally, past the window's end with its last
    // unit again, so the waits stay exact); the last partial group only
    // consumes.
    constexpr int R = kFtRing<FMT>;
    Unit<FMT> ring[R];
    float4 v0[kXb], v1[kXb];
    part(0, wa, wlen);
    wn = ntl * wlen;
    zero_rows();
    xload(0, 0, v0, v1);
#pragma unroll
    for (int d = 0; d < R; ++d) load(ring[d], d);
    for (;;) {
        xstore(cur, 0, v0, v1);
        convert_rest(cur, kXb * nthr);
        lds_barrier();
        // the first units are needed now anyway: waiting for every load here
        // (vmcnt(0)) leaves the steady loop below a clean entry state, so its
        // own waits are exact (one stage at a time)
        __builtin_amdgcn_s_waitcnt(0x0F70);
        int k = 0;
        for (; k + R <= wn; k += R) {
#pragma unroll
            for (int d = 0; d < R; ++d) {
                consume(ring[d]);
                __builtin_amdgcn_sched_barrier(0);
                load(ring[d], k + d + R);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int d = 0; d < R - 1; ++d)
            if (k + d < wn) consume(ring[d]);
        if (cur + 1 >= nwin) break;
        ++cur;
        part(cur, wa, wlen);
        wn = ntl * wlen;
        xload(cur, 0, v0, v1);
#pragma unroll
        for (int d = 0; d < R; ++d) load(ring[d], d);
        lds_barrier();  // every wave is done with the previous window
    }

    if (P == 1) {
        // whole tiles per wave: lanes 0..31 hold the high parts of tokens
        // 4g + v, lanes 32..63 the low parts of the same tokens
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            if (i < ntl) {
                const int64_t rr = r0 + 16 * (int64_t)(ts + i * nslots) + n;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float o = acc[i][v] + __shfl_xor(acc[i][v], 32);
                    const int t = 4 * g + v;
                    if (g < 2 && t < ntok && rr <= rl) y[(int64_t)t * M + rr] = o;
                }
            }
        }
    } else {
        // K split over the P waves of a tile: partials through LDS
        lds_barrier();
        float4* red = reinterpret_cast<float4*>(lds);
        red[wave * 64 + lane] = float4{acc[0][0], acc[0][1], acc[0][2], acc[0][3]};
        lds_barrier();
        const float* rf = reinterpret_cast<const float*>(lds);
        for (int it = tid; it < ntq * 128; it += nthr) {
            const int q = it >> 7, t = (it >> 4) & 7, nn = it & 15;
            const int64_t rr = r0 + 16 * (int64_t)q + nn;
            if (t < ntok && rr <= rl) {
                float o = 0.f;
                const float* hp = rf + (q * P * 64 + (t >> 2) * 16 + nn) * 4 + (t & 3);
#pragma unroll 4
                for (int p = 0; p < P; ++p) o += hp[p * 256] + hp[p * 256 + 128];
                y[(int64_t)t * M + rr] = o;
            }
        }
    }
}

template <int FMT, int TPW, int NS>
hipError_t launch_tpw(RowSegs<NS> sg, const float* x, int64_t K, int64_t n_tok, int nw, int rpw, int ntq, int P,
                      int ws, size_t lds, hipStream_t stream) {
    // workgroups per matrix: its rows in groups of rpw
    int64_t G = 0;
    for (int i = 0; i < NS; ++i) {
        sg.wg0[i] = sg.M[i] > 0 ? G : INT64_MAX;
        G += (sg.M[i] + rpw - 1) / rpw;
    }
    if (G > 0x7fffffff) return hipErrorNotSupported;
    if (query_only(kernel_name<Name_fewtok_kernel, FMT, TPW, NS>())) return hipSuccess;
    hipLaunchKernelGGL((fewtok_kernel<FMT, TPW, NS>), dim3((unsigned)G), dim3(64 * nw), lds, stream, sg, x, (int)K,
                       (int)n_tok, rpw, ntq, P, ws);
    return hipGetLastError();
}

int cu_count_ft() {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
        return 256;
    return v;
}

// M: rows of the row space (all segments)
template <int FMT, int NS>
hipError_t launch_f(const RowSegs<NS>& sg, const float* x, int64_t M, int64_t K, int64_t n_tok, hipStream_t stream) {
    if (n_tok < 2 || n_tok > 8 || K % 256 || M >= ((int64_t)1 << 30) || K >= ((int64_t)1 << 30))
        return hipErrorNotSupported;
    const int nsb = (int)(K / 256);
    const int64_t cus = cu_count_ft();
    // rows per workgroup: about M / #CU, at least 8
    int64_t G = (M + 7) / 8;
    if (G > cus) G = cus;
    int64_t rpw = (M + G - 1) / G;
    int ntq = (int)((rpw + 15) / 16);
    // Selection (MI355X sweeps against the few-token kernel of multitok.hip):
    // this kernel pays a workgroup-wide conversion of X per window, which
    // takes a few tiles per workgroup to amortize: it is taken from two tiles
    // per workgroup with K >= 4096 (Q4_K-style: any K) and for very tall
    // matrices (more tiles than waves); other shapes go to the other kernel.
    // The formats without that other kernel (the 5-bit ones, Q6_K, Q2_K,
    // MXFP4, q1_0) take this
    // one for every shape, a single tile with K split over up to 16 waves.
    constexpr bool only = kFtQ5<FMT> || kFtSub16<FMT> || FMT == LW_MXFP4 || FMT == LW_Q1_0;
    const bool take = only || ntq > kFtMaxWaves || (ntq >= 2 && (K >= 4096 || FMT == LW_Q4_K));
    if (!take) return hipErrorNotSupported;
    int nw, P, tpw;
    // tiles per wave at most (the 5-bit formats, which hold more per unit: 2)
    constexpr int max_tpw = kFtQ5<FMT> ? 2 : kFtMaxTpw;
    if (ntq > kFtMaxWaves) {
        // more tiles than waves: each wave owns whole tiles
        nw = kFtMaxWaves;
        P = 1;
        tpw = (ntq + nw - 1) / nw;
        if (tpw > max_tpw) {
            rpw = 16 * kFtMaxWaves * max_tpw;
            ntq = kFtMaxWaves * max_tpw;
            tpw = max_tpw;
        }
    } else {
        // waves split K: P parts per tile, preferring a P that divides the
        // super-blocks of a row
        const int pmax = kFtMaxWaves / ntq;
        P = pmax;
        for (int c = pmax; c >= (pmax + 1) / 2; --c)
            if (nsb % c == 0) {
                P = c;
                break;
            }
        nw = ntq * P;
        tpw = 1;
    }
    int ws = P * (kFtWinSB / P);
    if (ws > nsb) ws = nsb;
    size_t lds = (size_t)ws * 8 * 1024;  // the A slices of a window
    if (lds < (size_t)nw * 1024) lds = (size_t)nw * 1024;
    const int tp = tpw <= 1 ? 1 : tpw <= 2 ? 2 : 4;
    switch (tp) {
    case 1: return launch_tpw<FMT, 1, NS>(sg, x, K, n_tok, nw, (int)rpw, ntq, P, ws, lds, stream);
    case 2: return launch_tpw<FMT, 2, NS>(sg, x, K, n_tok, nw, (int)rpw, ntq, P, ws, lds, stream);
    default:
        if constexpr (max_tpw < 4)
            return hipErrorNotSupported;  // not reached: tpw <= max_tpw
        else
            return launch_tpw<FMT, 4, NS>(sg, x, K, n_tok, nw, (int)rpw, ntq, P, ws, lds, stream);
    }
}

template <int FMT>
hipError_t launch_one(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                      const Planes& p, hipStream_t stream) {
    RowSegs<1> sg;
    sg.W[0] = W;
    sg.y[0] = y;
    sg.off1[0] = p.off1;
    sg.off2[0] = p.off2;
    sg.off3[0] = p.off3;
    sg.start[0] = 0;
    sg.M[0] = M;
    return launch_f<FMT, 1>(sg, x, M, K, n_tok, stream);
}

template <int FMT, int NS>
hipError_t launch_segs(int n, const uint8_t* const* W, float* const* y, const int64_t* M, const float* x, int64_t K,
                       int64_t n_tok, hipStream_t stream) {
    RowSegs<NS> sg;
    int64_t tot = 0;
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
        if (used) tot += M[i];
    }
    return launch_f<FMT, NS>(sg, x, tot, K, n_tok, stream);
}

template <int FMT>
hipError_t launch_multi_ft(int n, const uint8_t* const* W, float* const* y, const int64_t* M, const float* x,
                           int64_t K, int64_t n_tok, hipStream_t stream) {
    if (n <= 2) return launch_segs<FMT, 2>(n, W, y, M, x, K, n_tok, stream);
    return launch_segs<FMT, kMaxSegs>(n, W, y, M, x, K, n_tok, stream);
}

}  // namespace

hipError_t launch_fewtok(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                         const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_one<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_one<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_one<LW_Q4_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_0: return launch_one<LW_Q5_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_1: return launch_one<LW_Q5_1>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q5_K: return launch_one<LW_Q5_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_MXFP4: return launch_one<LW_MXFP4>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q6_K: return launch_one<LW_Q6_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q2_K: return launch_one<LW_Q2_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q1_0: return launch_one<LW_Q1_0>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorNotSupported;
    }
}

hipError_t launch_fewtok_multi(int fmt, int n, const uint8_t* const* W, float* const* y, const int64_t* M,
                               const float* x, int64_t K, int64_t n_tok, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_multi_ft<LW_Q4_0>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q4_K: return launch_multi_ft<LW_Q4_K>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q4_1: return launch_multi_ft<LW_Q4_1>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q5_0: return launch_multi_ft<LW_Q5_0>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q5_1: return launch_multi_ft<LW_Q5_1>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q5_K: return launch_multi_ft<LW_Q5_K>(n, W, y, M, x, K, n_tok, stream);
    case LW_MXFP4: return launch_multi_ft<LW_MXFP4>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q6_K: return launch_multi_ft<LW_Q6_K>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q2_K: return launch_multi_ft<LW_Q2_K>(n, W, y, M, x, K, n_tok, stream);
    case LW_Q1_0: return launch_multi_ft<LW_Q1_0>(n, W, y, M, x, K, n_tok, stream);
    default: return hipErrorNotSupported;
    }
}

}  // namespace lw
