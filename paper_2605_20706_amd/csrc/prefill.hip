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
};

// Tiled kernel: a workgroup computes kBM weight rows x kBN tokens with four
// waves, wave (wm, wn) owning rows 64*wm .. +64 and tokens kTT*16*wn .. as
// 4 x kTT tiles of 16 x 16. Roles in D = A . B: A is X (16 tokens x one
// 32-element block), B the decoded codes (one block x 16 weight rows), so lane
// l holds D[4*(l/16) + v][l % 16] = (token 4*(l/16) + v, weight row l % 16) and
// one (c1, c2) pair per row tile and block serves its four outputs.
//
// K advances in stages of kKB blocks. Per stage the workgroup converts the X
// slab (kBN tokens x 32*kKB values) to hi/lo bf16 plus block sums, and the
// (c1, c2) coefficients of its kBM rows, into one of two LDS buffers (one
// barrier per stage). Each wave loads the codes of its own 64 rows directly
// into registers, two stages ahead. Consecutive workgroups take consecutive
// token tiles of the same rows, so a weight tile is read from HBM once and
// reused from L2 by the other token tiles.
constexpr int kBM = 128, kTT = 2, kBN = 32 * kTT, kKB = 2, kGT = 256;

struct GemmLds {
    // per buffer: xh, xl [kKB][4][kBN] x 16 B; xs [kKB][kBN] floats; cf [kKB][kBM] float2
    static constexpr int kX = kKB * 4 * kBN;                 // bf16x8 entries per half
    static constexpr size_t kBuf = (size_t)2 * kX * 16 + (size_t)kKB * kBN * 4 + (size_t)kKB * kBM * 8;
    static constexpr size_t kBytes = 2 * kBuf;
};

template <int FMT>
__global__ void __launch_bounds__(kGT) __attribute__((amdgpu_waves_per_eu(2, 2)))
    gemm_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                int64_t K, int64_t N, int64_t off1, int64_t off2) {
    using T = MF<FMT>;
    using Word = decltype(T::code_word(nullptr, 0, 0, 0, 0));
    extern __shared__ bf16x8 smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;
    const int i16 = lane & 15, s4 = lane >> 4;
    const int64_t ntt = (N + kBN - 1) / kBN;
    const int64_t row0 = (int64_t)(blockIdx.x / ntt) * kBM;
    const int64_t tok0 = (int64_t)(blockIdx.x % ntt) * kBN;
    const uint32_t K32 = (uint32_t)K;
    const int nst = (int)(K / (32 * kKB));  // K is a multiple of 256: whole stages

    auto buf_xh = [&](int bf) { return smem + (size_t)bf * (GemmLds::kBuf / 16); };
    auto buf_xl = [&](int bf) { return buf_xh(bf) + GemmLds::kX; };
    auto buf_xs = [&](int bf) { return reinterpret_cast<float*>(buf_xh(bf) + 2 * GemmLds::kX); };
    auto buf_cf = [&](int bf) { return reinterpret_cast<float2*>(buf_xs(bf) + kKB * kBN); };

    // weight rows of this lane (B operand column), clamped; stores are masked
    uint64_t wrow[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int64_t r = row0 + 64 * wm + 16 * rt + i16;
        wrow[rt] = (uint64_t)(r < M ? r : M - 1);
    }
    auto load_codes = [&](Word (*cw)[kKB], int st) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int b = 0; b < kKB; ++b) cw[rt][b] = T::code_word(W, wrow[rt], K32, st * kKB + b, s4);
    };

    // stage producers: X items (block, token, slice) and coefficient items (block, row)
    constexpr int kXI = kKB * kBN * 4 / kGT;  // 4
    float4 xa[kXI], xb[kXI];
    uint32_t sraw[4];  // raw scale data of this thread's coefficient item
    const int ci_r = tid % kBM, ci_b = tid / kBM;
    const int64_t ci_row = row0 + ci_r < M ? row0 + ci_r : M - 1;
    auto fetch = [&](int st) {
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
        T::load_scale(W, off1, off2, (uint64_t)ci_row, K32, st * kKB + ci_b, sraw);
    };
    auto commit = [&](int bf, int st) {
        bf16x8* xh = buf_xh(bf);
        bf16x8* xl = buf_xl(bf);
        float* xs = buf_xs(bf);
#pragma unroll
        for (int i = 0; i < kXI; ++i) {
            const int it = tid + i * kGT;
            const int sl = it & 3, t = (it >> 2) % kBN, b = (it >> 2) / kBN;
            const float v[8] = {xa[i].x, xa[i].y, xa[i].z, xa[i].w, xb[i].x, xb[i].y, xb[i].z, xb[i].w};
            bf16x8 h, l;
            float sum = split_bf16x8(v, &h, &l);
            xh[(b * 4 + sl) * kBN + t] = h;
            xl[(b * 4 + sl) * kBN + t] = l;
            if constexpr (T::kSums) {
                sum += dpp_move<0xB1>(sum);  // the 4 slices of (block, token) are one lane quad
                sum += dpp_move<0x4E>(sum);
                if (sl == 0) xs[b * kBN + t] = sum;
            }
        }
        float c1, c2;
        T::coef_raw(sraw, st * kKB + ci_b, &c1, &c2);
        buf_cf(bf)[ci_b * kBM + ci_r] = make_float2(c1, c2);
    };

    f32x4 acc[4][kTT];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int tt = 0; tt < kTT; ++tt) acc[rt][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int bf, Word (*cw)[kKB]) {
        const bf16x8* xh = buf_xh(bf);
        const bf16x8* xl = buf_xl(bf);
        const float* xs = buf_xs(bf);
        const float2* cf = buf_cf(bf);
#pragma unroll
        for (int b = 0; b < kKB; ++b) {
            bf16x8 ah[kTT], al[kTT];
            f32x4 sm[kTT];
#pragma unroll
            for (int tt = 0; tt < kTT; ++tt) {
                const int t = 16 * kTT * wn + 16 * tt;
                ah[tt] = xh[(b * 4 + s4) * kBN + t + i16];
                al[tt] = xl[(b * 4 + s4) * kBN + t + i16];
                if constexpr (T::kSums) sm[tt] = *reinterpret_cast<const f32x4*>(&xs[b * kBN + t + 4 * s4]);
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                const bf16x8 bw = T::decode(cw[rt][b]);
                const float2 c = cf[b * kBM + 64 * wm + 16 * rt + i16];
#pragma unroll
                for (int tt = 0; tt < kTT; ++tt) {
                    f32x4 p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[tt], bw, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[tt], bw, p, 0, 0, 0);
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float o = __builtin_fmaf(c.x, p[v], acc[rt][tt][v]);
                        if constexpr (T::kSums) o = __builtin_fmaf(c.y, sm[tt][v], o);
                        acc[rt][tt][v] = o;
                    }
                }
            }
        }
    };

    Word cwA[4][kKB], cwB[4][kKB];
    load_codes(cwA, 0);
    if (nst > 1) load_codes(cwB, 1);
    fetch(0);
    commit(0, 0);
    if (nst > 1) fetch(1);
    __syncthreads();
    // stages in pairs (nst is even): codes of stage st are in cwA for even st, cwB for odd st
    for (int st = 0; st < nst; st += 2) {
        compute(0, cwA);
        if (st + 2 < nst) load_codes(cwA, st + 2);
        if (st + 1 < nst) {
            commit(1, st + 1);
            if (st + 2 < nst) fetch(st + 2);
        }
        __syncthreads();
        if (st + 1 < nst) {
            compute(1, cwB);
            if (st + 3 < nst) load_codes(cwB, st + 3);
            if (st + 2 < nst) {
                commit(0, st + 2);
                if (st + 3 < nst) fetch(st + 3);
            }
            __syncthreads();
        }
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
