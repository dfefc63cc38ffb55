// Multi-token product on the matrix cores (n_tok >= 2).
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k]. With two or more tokens the
// product is a contraction over K with a token dimension, so it runs on
// v_mfma_f32_16x16x32_bf16 (Sec. 3.2: matrix multiplication tiles through
// shared memory and uses the cooperative matrix instructions of the device;
// Sec. 3.3: quantized blocks are dequantized on the way in and each decoded
// tile is reused for every token of the workgroup).
//
// Precision. One MFMA K-step is one 32-element block. The A operand holds
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
// The B operand in LDS uses the same order of k.
//
// Workgroup = G row groups x S K-splits waves. Wave (g, q) computes 16 rows x
// 16*NTT tokens over the K range of split q; K advances in stages of KB
// blocks per split. Per stage the workgroup converts its X slab to hi/lo bf16
// into LDS and stages the block coefficients of its rows; codes come straight
// from HBM, two stages ahead. LDS is double-buffered: one barrier per stage.
// With S > 1 the split partials are summed through LDS at the end.
#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));


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
        // byte b -> 16-bit lane: (q_b0 | q_b1 << 16), (q_b2 | q_b3 << 16)
        const uint32_t l01 = __builtin_amdgcn_perm(0u, lo, 0x0c010c00u) | 0x43004300u;
        const uint32_t l23 = __builtin_amdgcn_perm(0u, lo, 0x0c030c02u) | 0x43004300u;
        const uint32_t h01 = __builtin_amdgcn_perm(0u, hi, 0x0c010c00u) | 0x43004300u;
        const uint32_t h23 = __builtin_amdgcn_perm(0u, hi, 0x0c030c02u) | 0x43004300u;
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = {l01, l23, h01, h23};
        return __builtin_bit_cast(bf16x8, v);
    }
    __device__ static int x_first(int s, int half) { return half ? 16 + 4 * s : 4 * s; }
    // coefficients (c1, c2) of the block: y += c1 * P + c2 * S
    __device__ static void coef(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K, int blk,
                                float* c1, float* c2) {
        if constexpr (FMT == LW_Q4_0) {
            const float d = half_bits_to_float(
                *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk)));
            *c1 = d;
            *c2 = -136.0f * d;
        } else {
            const uint64_t S = row * (K / 256u) + (uint32_t)(blk >> 3);
            const int j = blk & 7;
            const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * S);
            const uint64_t lo = (uint64_t)rec[0] | ((uint64_t)rec[1] << 32);
            const uint64_t hi = (uint64_t)rec[1] | ((uint64_t)rec[2] << 32);
            const uint32_t dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * S);
            const float ds = half_bits_to_float(dd & 0xFFFFu) * (float)((uint32_t)(lo >> (6 * j)) & 63u);
            const float dm = half_bits_to_float(dd >> 16) * (float)((uint32_t)(hi >> (16 + 6 * j)) & 63u);
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
    __device__ static void coef(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, int blk,
                                float* c1, float* c2) {
        *c1 = half_bits_to_float(
            *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk)));
        *c2 = 0.f;
    }
};

// Workgroup configuration: G x S waves; wave (g, q) computes RG row groups of
// 16 rows (rows 16*RG*g .. +16*RG) x NTT token tiles of 16 over the K range of
// split q; KB blocks of 32 per split per stage.
template <int RG, int NTT, int G, int S, int KB>
struct Cfg {
    static constexpr int kThreads = 64 * G * S;
    static constexpr int kRows = 16 * RG * G;
    static constexpr int kTok = 16 * NTT;
};

// Dynamic LDS of one launch (tk = tokens of the workgroup staged, <= kTok):
//   B hi, B lo: [2][S][KB][4 slices][tk] x 16 bytes
//   coefficients c1, c2: [2][S][KB][kRows] floats
//   block sums: [2][S][KB][tk] floats (4-bit formats)
template <int RG, int NTT, int G, int S, int KB>
struct Lds {
    int tk, nb, nc, ns;
    __host__ __device__ Lds(int tk_) : tk(tk_), nb(S * KB * 4 * tk_), nc(S * KB * 16 * RG * G), ns(S * KB * tk_) {}
    __host__ __device__ size_t bytes() const { return (size_t)2 * (2 * nb * 16 + 2 * nc * 4 + ns * 4); }
};

template <int FMT, int RG, int NTT, int G, int S, int KB>
__global__ void __launch_bounds__(64 * G * S)
    mfma_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                int64_t K, int64_t N, int64_t off1, int64_t off2) {
    using T = MF<FMT>;
    using C = Cfg<RG, NTT, G, S, KB>;
    using Word = decltype(T::code_word(nullptr, 0, 0, 0, 0));
    extern __shared__ bf16x8 smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = wave % G, q = wave / G;
    const int i16 = lane & 15, s4 = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.x * C::kRows;
    const int64_t tok0 = (int64_t)blockIdx.y * C::kTok;
    const uint32_t K32 = (uint32_t)K;
    const int nblk = (int)(K / 32);
    const int nst = (nblk + S * KB - 1) / (S * KB);  // split q owns blocks [q*nst*KB, (q+1)*nst*KB)
    const int tk = (int)((N - tok0) < C::kTok ? (N - tok0) : C::kTok);  // real tokens of the workgroup
    const Lds<RG, NTT, G, S, KB> L(tk);
    bf16x8* bhi = smem;                                       // [2][nb]
    bf16x8* blo = smem + 2 * L.nb;                            // [2][nb]
    float* cf1 = reinterpret_cast<float*>(smem + 4 * L.nb);  // [2][nc]
    float* cf2 = cf1 + 2 * L.nc;                              // [2][nc]
    float* bsum = cf2 + 2 * L.nc;                             // [2][ns]

    uint64_t arow[RG];
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
        const int64_t r = row0 + 16 * (RG * g + rg) + i16;
        arow[rg] = (uint64_t)(r < M ? r : M - 1);
    }

    // ---- stage producers: codes (registers), X and coefficients (registers -> LDS) ----
    auto load_codes = [&](Word (*cw)[KB], int st) {
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int b = 0; b < KB; ++b) {
                const int blk = (q * nst + st) * KB + b;
                cw[rg][b] = blk < nblk ? T::code_word(W, arow[rg], K32, blk, s4) : Word(0);
            }
    };
    constexpr int kXI = (S * KB * 4 * C::kTok + C::kThreads - 1) / C::kThreads;  // X items per thread (max)
    constexpr int kCI = (S * KB * C::kRows + C::kThreads - 1) / C::kThreads;    // coefficient items per thread
    const int nxi = S * KB * tk * 4;  // X items of a stage: (split, block, token, slice)
    float4 xa[kXI], xb[kXI];
    float c1r[kCI], c2r[kCI];
    auto fetch = [&](int st) {  // global loads of stage st into registers
#pragma unroll
        for (int i = 0; i < kXI; ++i) {
            const int it = tid + i * C::kThreads;
            const int s = it & 3, t = (it >> 2) % tk, qb = (it >> 2) / tk;
            const int b = qb % KB, qq = qb / KB;
            const int blk = (qq * nst + st) * KB + b;
            // loads stay in bounds for dead items (element 0 of X); their values are dropped
            const bool ok = it < nxi && blk < nblk;
            const float* xp = x + (ok ? (tok0 + t) * K + 32 * (int64_t)blk : 0);
            const float4 u0 = *reinterpret_cast<const float4*>(xp + (ok ? T::x_first(s, 0) : 0));
            const float4 u1 = *reinterpret_cast<const float4*>(xp + (ok ? T::x_first(s, 1) : 0));
            const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
            xa[i] = ok ? u0 : z;
            xb[i] = ok ? u1 : z;
        }
#pragma unroll
        for (int i = 0; i < kCI; ++i) {
            const int it = tid + i * C::kThreads;
            const int r = it % C::kRows, qb = it / C::kRows;
            const int b = qb % KB, qq = qb / KB;
            const int blk = (qq * nst + st) * KB + b;
            const int64_t rr = row0 + r;
            c1r[i] = c2r[i] = 0.f;
            if (it < L.nc && rr < M && blk < nblk) T::coef(W, off1, off2, (uint64_t)rr, K32, blk, &c1r[i], &c2r[i]);
        }
    };
    auto commit = [&](int buf) {  // registers -> LDS buffer buf
#pragma unroll
        for (int i = 0; i < kXI; ++i) {
            const int it = tid + i * C::kThreads;
            if (i * C::kThreads >= ((nxi + 63) & ~63)) break;  // whole waves only (DPP below)
            const bool live = it < nxi;
            const int s = it & 3, t = (it >> 2) % tk, qb = (it >> 2) / tk;
            const float v[8] = {xa[i].x, xa[i].y, xa[i].z, xa[i].w, xb[i].x, xb[i].y, xb[i].z, xb[i].w};
            bf16x8 h, l;
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                h[e] = (__bf16)v[e];
                const float hf = (float)h[e];
                l[e] = (__bf16)(v[e] - hf);
                sum += hf + (float)l[e];
            }
            if (live) {
                const int idx = (qb * 4 + s) * tk + t;  // qb = split * KB + block
                bhi[buf * L.nb + idx] = h;
                blo[buf * L.nb + idx] = l;
            }
            if constexpr (T::kSums) {
                sum += dpp_move<0xB1>(sum);  // the 4 slices of (split, block, token): one lane quad
                sum += dpp_move<0x4E>(sum);
                if (live && s == 0) bsum[buf * L.ns + qb * tk + t] = sum;
            }
        }
#pragma unroll
        for (int i = 0; i < kCI; ++i) {
            const int it = tid + i * C::kThreads;
            if (it < L.nc) {
                cf1[buf * L.nc + it] = c1r[i];
                cf2[buf * L.nc + it] = c2r[i];
            }
        }
    };

    f32x4 acc[RG][NTT];
#pragma unroll
    for (int rg = 0; rg < RG; ++rg)
#pragma unroll
        for (int t = 0; t < NTT; ++t) acc[rg][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    Word cw0[RG][KB], cw1[RG][KB], cw2[RG][KB];  // codes of stages st, st+1, st+2
    load_codes(cw0, 0);
    fetch(0);
    if (nst > 1) load_codes(cw1, 1);
    commit(0);
    if (nst > 1) fetch(1);
    __syncthreads();

    for (int st = 0; st < nst; ++st) {
        const int buf = st & 1;
        if (st + 2 < nst) load_codes(cw2, st + 2);
        const bf16x8* Bh = bhi + buf * L.nb;
        const bf16x8* Bl = blo + buf * L.nb;
#pragma unroll
        for (int b = 0; b < KB; ++b) {
            const int qb = q * KB + b;
            bf16x8 a[RG];
            f32x4 c1[RG], c2[RG];
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                a[rg] = T::decode(cw0[rg][b]);
                const int cbase = buf * L.nc + qb * C::kRows + 16 * (RG * g + rg) + 4 * s4;
                c1[rg] = *reinterpret_cast<const f32x4*>(&cf1[cbase]);
                if constexpr (T::kSums) c2[rg] = *reinterpret_cast<const f32x4*>(&cf2[cbase]);
            }
#pragma unroll
            for (int t = 0; t < NTT; ++t) {
                int col = 16 * t + i16;
                col = col < tk ? col : tk - 1;  // padded columns reuse a real one; never stored
                const bf16x8 bh = Bh[(qb * 4 + s4) * tk + col];
                const bf16x8 bl = Bl[(qb * 4 + s4) * tk + col];
                float sm = 0.f;
                if constexpr (T::kSums) sm = bsum[buf * L.ns + qb * tk + col];
#pragma unroll
                for (int rg = 0; rg < RG; ++rg) {
                    f32x4 p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rg], bh, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rg], bl, p, 0, 0, 0);
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float o = __builtin_fmaf(c1[rg][v], p[v], acc[rg][t][v]);
                        if constexpr (T::kSums) o = __builtin_fmaf(c2[rg][v], sm, o);
                        acc[rg][t][v] = o;
                    }
                }
            }
        }
        if (st + 1 < nst) {
            commit(buf ^ 1);  // buffer buf^1 was last read before the previous barrier
            if (st + 2 < nst) fetch(st + 2);
        }
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int b = 0; b < KB; ++b) {
                cw0[rg][b] = cw1[rg][b];
                cw1[rg][b] = cw2[rg][b];
            }
        __syncthreads();
    }

    // ---- sum the K-split partials and store ----
    // lane holds rows 16*(RG*g + rg) + 4*s4 + v, token column 16t + i16
    if constexpr (S > 1) {
        float* red = reinterpret_cast<float*>(smem);  // S x kRows x kTok floats
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int t = 0; t < NTT; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    red[(q * C::kRows + 16 * (RG * g + rg) + 4 * s4 + v) * C::kTok + 16 * t + i16] = acc[rg][t][v];
        __syncthreads();
        for (int it = tid; it < C::kRows * C::kTok; it += C::kThreads) {
            const int r = it / C::kTok, t = it % C::kTok;
            const int64_t rr = row0 + r;
            if (rr < M && t < tk) {
                float o = 0.f;
                for (int qq = 0; qq < S; ++qq) o += red[(qq * C::kRows + r) * C::kTok + t];
                y[(tok0 + t) * M + rr] = o;
            }
        }
    } else {
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int t = 0; t < NTT; ++t) {
                const int tl = 16 * t + i16;
                if (tl >= tk) continue;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t rr = row0 + 16 * (RG * g + rg) + 4 * s4 + v;
                    if (rr < M) y[(tok0 + tl) * M + rr] = acc[rg][t][v];
                }
            }
    }
}

template <int FMT, int RG, int NTT, int G, int S, int KB>
hipError_t launch_cfg(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                      const Planes& p, hipStream_t stream) {
    using C = Cfg<RG, NTT, G, S, KB>;
    const int64_t gm = (M + C::kRows - 1) / C::kRows, gn = (n_tok + C::kTok - 1) / C::kTok;
    if (gm > 0x7fffffff || gn > 65535) return hipErrorInvalidConfiguration;
    const int tk = (int)(n_tok < C::kTok ? n_tok : C::kTok);
    size_t lds = Lds<RG, NTT, G, S, KB>(tk).bytes();
    const size_t red = (size_t)4 * S * C::kRows * C::kTok;  // split reduction reuses the buffer
    if (S > 1 && red > lds) lds = red;
    if (lds > (size_t)160 * 1024) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((mfma_kernel<FMT, RG, NTT, G, S, KB>), dim3((unsigned)gm, (unsigned)gn), dim3(C::kThreads),
                       lds, stream, W, x, y, M, K, n_tok, p.off1, p.off2);
    return hipGetLastError();
}

template <int FMT>
hipError_t launch_mfma(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                       const Planes& p, hipStream_t stream) {
    // up to 16 tokens: one token tile per wave, K split 4 ways so that enough
    // waves stream the weights; more tokens: 2 row groups x 4 token tiles per wave.
    if (n_tok <= 16) return launch_cfg<FMT, 1, 1, 2, 4, 8>(W, x, y, M, K, n_tok, p, stream);
    return launch_cfg<FMT, 2, 4, 4, 1, 4>(W, x, y, M, K, n_tok, p, stream);
}

}  // namespace

hipError_t launch_prefill(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                          int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_mfma<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_mfma<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_mfma<LW_Q8_0>(W, x, y, M, K, n_tok, p, stream);
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
