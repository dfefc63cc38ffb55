// Few-token product on the matrix cores: 2 <= n_tok <= 16 (batched decode).
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k] with the weights streamed from
// HBM once for all tokens (Sec. 2.1: decode; Sec. 3.3: codes dequantized
// directly into registers). The product is formed as D = X . W^T on
// v_mfma_f32_16x16x32_bf16: the A operand is X (16 token rows x one 32-element
// block), the B operand holds the codes of 16 weight rows. In the MFMA output
// layout lane l then owns D[4*(l/16) + v][l % 16], i.e. four tokens of weight
// row l % 16 -- the very row whose codes lane l loads -- so each lane applies
// its own row's block scale without any exchange.
//
// Precision: as on the prefill path -- B holds the exact bf16 of the biased
// 4-bit code 128 + q (Q4_0, Q4_K-style, Q4_1) or of the int8 code (Q8_0); X is split
// into bf16 high and low parts; per block, y += c1 * P + c2 * S with S the sum
// of the block's hi + lo values, so the bias cancels to float32 rounding.
//
// Workgroup: S waves, all on the same 16 weight rows, each on one K split.
// X (the real tokens only) is converted once per K tile into LDS as hi/lo
// bf16 plus block sums; codes and scales stream from HBM per lane, two steps
// of 4 blocks ahead, with no barrier inside a K tile. The split partials are
// summed through LDS at the end.
#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

// names of the kernel templates, for lw_kernel_name
struct Name_skinny_kernel {
    static constexpr const char* base = "skinny_kernel";
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kStep = 4;                      // blocks per prefetch step
constexpr int64_t kXLds = 96 * 1024;          // LDS for an X tile (hi, lo and block sums)

template <int FMT>
struct SK;

// 4-bit formats. Codes: word s of the block's 16 bytes (elements 4s..4s+3 in the
// low nibbles, 16+4s..16+4s+3 in the high nibbles); B operand = 128 + q.
template <int FMT>
struct SK4 {
    static constexpr bool kSums = true;
    __device__ static uint32_t code(const uint8_t* W, uint64_t row, uint32_t K, int blk, int s) {
        return __builtin_nontemporal_load(
            reinterpret_cast<const uint32_t*>(W + row * (K / 2u) + 16u * (uint32_t)blk + 4u * s));
    }
    __device__ static bf16x8 decode(uint32_t w) {
        const uint32_t lo = opaque(w & 0x0F0F0F0Fu);
        const uint32_t hi = opaque((w >> 4) & 0x0F0F0F0Fu);
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = {__builtin_amdgcn_perm(0u, lo, 0x0c010c00u) | 0x43004300u,
                         __builtin_amdgcn_perm(0u, lo, 0x0c030c02u) | 0x43004300u,
                         __builtin_amdgcn_perm(0u, hi, 0x0c010c00u) | 0x43004300u,
                         __builtin_amdgcn_perm(0u, hi, 0x0c030c02u) | 0x43004300u};
        return __builtin_bit_cast(bf16x8, v);
    }
    __device__ static int x_first(int s, int half) { return half ? 16 + 4 * s : 4 * s; }
    // raw scale data of one step (4 blocks starting at a multiple of 4) of a row
    struct Raw {
        uint32_t a, b, c, d;
    };
    __device__ static Raw load_raw(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K, int blk) {
        Raw r;
        if constexpr (FMT == LW_Q4_0) {
            const uint2 v = *reinterpret_cast<const uint2*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk));
            r.a = v.x;
            r.b = v.y;
            r.c = r.d = 0;
        } else if constexpr (FMT == LW_Q4_1) {
            const uint4 v = *reinterpret_cast<const uint4*>(W + off1 + 4 * (row * (K / 32u) + (uint32_t)blk));
            r.a = v.x;  // {d, m} of the step's 4 blocks
            r.b = v.y;
            r.c = v.z;
            r.d = v.w;
        } else {
            const uint64_t Sb = row * (K / 256u) + (uint32_t)(blk >> 3);
            const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * Sb);
            r.a = rec[0];
            r.b = rec[1];
            r.c = rec[2];
            r.d = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * Sb);
        }
        return r;
    }
    // coefficients of block blk (its index within the step is blk & 3): y += c1*P + c2*S
    __device__ static void coef(const Raw& r, int blk, float* c1, float* c2) {
        if constexpr (FMT == LW_Q4_0) {
            const int i = blk & 3;
            const uint32_t h = (i < 2 ? r.a : r.b) >> (16 * (i & 1));
            const float d = half_bits_to_float(h & 0xFFFFu);
            *c1 = d;
            *c2 = -136.0f * d;
        } else if constexpr (FMT == LW_Q4_1) {
            const int i = blk & 3;
            const uint32_t dm = i == 0 ? r.a : i == 1 ? r.b : i == 2 ? r.c : r.d;
            const float d = half_bits_to_float(dm & 0xFFFFu);
            *c1 = d;
            *c2 = __builtin_fmaf(-128.0f, d, half_bits_to_float(dm >> 16));  // m - 128 d
        } else {
            const int j = blk & 7;
            const uint64_t lo = (uint64_t)r.a | ((uint64_t)r.b << 32);
            const uint64_t hi = (uint64_t)r.b | ((uint64_t)r.c << 32);
            const float ds = half_bits_to_float(r.d & 0xFFFFu) * (float)((uint32_t)(lo >> (6 * j)) & 63u);
            const float dm = half_bits_to_float(r.d >> 16) * (float)((uint32_t)(hi >> (16 + 6 * j)) & 63u);
            *c1 = ds;
            *c2 = -__builtin_fmaf(128.0f, ds, dm);
        }
    }
};
template <>
struct SK<LW_Q4_0> : SK4<LW_Q4_0> {};
template <>
struct SK<LW_Q4_K> : SK4<LW_Q4_K> {};
template <>
struct SK<LW_Q4_1> : SK4<LW_Q4_1> {};

template <>
struct SK<LW_Q8_0> {
    static constexpr bool kSums = false;
    __device__ static uint64_t code(const uint8_t* W, uint64_t row, uint32_t K, int blk, int s) {
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
    struct Raw {
        uint32_t a, b;
    };
    __device__ static Raw load_raw(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, int blk) {
        const uint2 v = *reinterpret_cast<const uint2*>(W + off1 + 2 * (row * (K / 32u) + (uint32_t)blk));
        return {v.x, v.y};
    }
    __device__ static void coef(const Raw& r, int blk, float* c1, float* c2) {
        const int i = blk & 3;
        const uint32_t h = (i < 2 ? r.a : r.b) >> (16 * (i & 1));
        *c1 = half_bits_to_float(h & 0xFFFFu);
        *c2 = 0.f;
    }
};

template <int FMT, int S>
__global__ void __launch_bounds__(64 * S)
    skinny_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                  int64_t K, int ntok, int KT, int64_t off1, int64_t off2) {
    using T = SK<FMT>;
    using Word = decltype(T::code(nullptr, 0, 0, 0, 0));
    using Raw = typename T::Raw;
    extern __shared__ bf16x8 smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, q = tid >> 6;  // wave = K split
    const int i16 = lane & 15, s4 = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.x * 16;
    const uint32_t K32 = (uint32_t)K;
    const int64_t rr = row0 + i16;
    const uint64_t brow = (uint64_t)(rr < M ? rr : M - 1);  // this lane's weight row (B column)
    const int tcl = i16 < ntok ? i16 : ntok - 1;            // this lane's token row of A (clamped)

    const int kbt = KT / 32;                 // blocks per K tile
    const int nbq = ((kbt + S - 1) / S + kStep - 1) / kStep * kStep;  // blocks per split, whole steps
    const int nstp = (nbq + kStep - 1) / kStep;
    bf16x8* xh = smem;                                   // [kbt][4][ntok]
    bf16x8* xl = smem + kbt * 4 * ntok;                  // [kbt][4][ntok]
    float* bs = reinterpret_cast<float*>(xl + kbt * 4 * ntok);  // [kbt][ntok] block sums

    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int64_t k0 = 0; k0 < K; k0 += KT) {
        const int kt = (int)((K - k0) < KT ? (K - k0) : KT);
        const int nbt = kt / 32;
        const int bq0 = q * nbq;                          // first block (within the tile) of this split
        const int bq1 = (bq0 + nbq) < nbt ? (bq0 + nbq) : nbt;
        const int gb0 = (int)(k0 / 32);                   // first block of the tile in the row
        // step loads: codes of 4 blocks and their scale data
        auto load_step = [&](Word* cw, Raw& raw, int st) {
            const int b0 = bq0 + st * kStep;
#pragma unroll
            for (int b = 0; b < kStep; ++b) {
                const int bb = b0 + b < bq1 ? b0 + b : bq1 - 1;  // clamped; masked in compute
                cw[b] = T::code(W, brow, K32, gb0 + bb, s4);
            }
            raw = T::load_raw(W, off1, off2, brow, K32, gb0 + (b0 < bq1 ? b0 : bq1 - 1) / kStep * kStep);
        };
        Word cw0[kStep], cw1[kStep], cw2[kStep];
        Raw r0, r1, r2;
        if (bq0 < bq1) {
            load_step(cw0, r0, 0);
            if (nstp > 1) load_step(cw1, r1, 1);
        }
        // X tile -> LDS: items (block, token, slice), all threads
        if (k0) __syncthreads();  // the previous tile is consumed
        const int nit = nbt * ntok * 4;
        for (int it0 = 0; it0 < nit; it0 += 64 * S) {
            const int it = it0 + tid;
            const bool live = it < nit;
            const int s = it & 3, t = (it >> 2) % ntok, b = (it >> 2) / ntok;
            const float* xp = x + (live ? (int64_t)t * K + k0 + 32 * b : 0);
            const float4 u0 = *reinterpret_cast<const float4*>(xp + (live ? T::x_first(s, 0) : 0));
            const float4 u1 = *reinterpret_cast<const float4*>(xp + (live ? T::x_first(s, 1) : 0));
            const float v[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
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
                xh[(b * 4 + s) * ntok + t] = h;
                xl[(b * 4 + s) * ntok + t] = l;
            }
            if constexpr (T::kSums) {
                sum += dpp_move<0xB1>(sum);  // the 4 slices of (block, token) are a lane quad
                sum += dpp_move<0x4E>(sum);
                if (live && s == 0) bs[b * ntok + t] = sum;
            }
        }
        __syncthreads();

        for (int st = 0; st < nstp && bq0 < bq1; ++st) {
            if (st + 2 < nstp) load_step(cw2, r2, st + 2);
            const int b0 = bq0 + st * kStep;
#pragma unroll
            for (int b = 0; b < kStep; ++b) {
                const int bb = b0 + b;
                if (bb < bq1) {  // uniform across the wave
                    const bf16x8 a_h = xh[(bb * 4 + s4) * ntok + tcl];
                    const bf16x8 a_l = xl[(bb * 4 + s4) * ntok + tcl];
                    const bf16x8 bw = T::decode(cw0[b]);
                    f32x4 p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_h, bw, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_l, bw, p, 0, 0, 0);
                    float c1, c2;
                    T::coef(r0, gb0 + bb, &c1, &c2);
                    f32x4 sm = {0.f, 0.f, 0.f, 0.f};
                    if constexpr (T::kSums) {
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const int tt = 4 * s4 + v;
                            sm[v] = bs[bb * ntok + (tt < ntok ? tt : ntok - 1)];
                        }
                    }
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float o = __builtin_fmaf(c1, p[v], acc[v]);
                        if constexpr (T::kSums) o = __builtin_fmaf(c2, sm[v], o);
                        acc[v] = o;
                    }
                }
            }
#pragma unroll
            for (int b = 0; b < kStep; ++b) {
                cw0[b] = cw1[b];
                cw1[b] = cw2[b];
            }
            r0 = r1;
            r1 = r2;
        }
    }

    // sum the split partials: lane holds tokens 4*s4 + v of weight row i16
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);  // [S][16 tokens][16 rows]
#pragma unroll
    for (int v = 0; v < 4; ++v) red[(q * 16 + 4 * s4 + v) * 16 + i16] = acc[v];
    __syncthreads();
    for (int it = tid; it < 256; it += 64 * S) {
        const int t = it >> 4, r = it & 15;
        if (t < ntok && row0 + r < M) {
            float o = 0.f;
            for (int qq = 0; qq < S; ++qq) o += red[(qq * 16 + t) * 16 + r];
            y[(int64_t)t * M + row0 + r] = o;
        }
    }
}

template <int FMT, int S>
hipError_t launch_s(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                    const Planes& p, hipStream_t stream) {
    // K tile: as many 32-element blocks as fit the X budget (32 * ntok bytes... per element 4 bytes
    // of hi/lo plus 4 bytes of block sum per 32), a multiple of 32 * 4 * S elements when tiled.
    const int64_t per_elem = 4 * n_tok;                    // hi + lo bf16 per element and token
    int64_t KT = kXLds / (per_elem + (4 * n_tok + 31) / 32);
    const int64_t unit = 32 * kStep * S;
    KT = KT / unit * unit;
    if (KT < unit) KT = unit;
    if (KT >= K) KT = K;
    const int64_t kbt = KT / 32;
    size_t lds = (size_t)(kbt * 4 * n_tok * 16 * 2 + kbt * n_tok * 4);
    if (lds < (size_t)S * 256 * 4) lds = (size_t)S * 256 * 4;  // final split reduction
    const int64_t grid = (M + 15) / 16;
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (query_only(kernel_name<Name_skinny_kernel, FMT, S>())) return hipSuccess;
    hipLaunchKernelGGL((skinny_kernel<FMT, S>), dim3((unsigned)grid), dim3(64 * S), lds, stream, W, x, y, M, K,
                       (int)n_tok, (int)KT, p.off1, p.off2);
    return hipGetLastError();
}

}  // namespace

bool skinny_supported(int fmt) { return fmt == LW_Q4_0 || fmt == LW_Q4_K || fmt == LW_Q4_1 || fmt == LW_Q8_0; }

hipError_t launch_skinny(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                         const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_s<LW_Q4_0, 4>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_s<LW_Q4_K, 4>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_s<LW_Q4_1, 4>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_s<LW_Q8_0, 4>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
