// Few-token product on the matrix cores for the 4-bit formats (2 <= n_tok <= 16).
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k]: the decode product of Sec. 2.1
// for a small batch of tokens, with the weights streamed from HBM exactly once
// and dequantized in registers (Sec. 3.3). The contraction runs on
// v_mfma_f32_16x16x32_bf16 (D[16x16] += A[16x32] . B[32x16]).
//
// Operand mapping. Lane l = 16*g + n (g = l/16, n = l%16) loads the 16 code
// bytes of one whole 32-weight block: block 4s+g of weight row n, for step s
// (4 blocks = 128 columns). Word j of those bytes holds elements 4j..4j+3 (low
// nibbles) and 16+4j..16+4j+3 (high nibbles) of the block, which become the 8
// bf16 B values of the lane in MFMA j (j = 0..3). So in MFMA j the 32 K indices
// are quarter j of four different blocks (one per lane group g).
//
// To keep every block's scale separate, A is block-diagonal: A row i stands
// for (block i/4, token i%4) and holds X only in the K indices of its own
// block; all other entries are zero. Summed over j = 0..3, D[i][n] is then the
// dot product of token i%4 with block i/4 of row n. In the MFMA output layout
// lane l holds D[4g + v][n], v = 0..3: the four tokens of block 4s+g of row n,
// i.e. exactly the block whose codes (and scale) the lane loaded -- each lane
// applies its own block's scale with no data exchange, once per step.
//
// Precision (the same reading as the other matrix-core paths): B holds the
// exact bf16 of the biased code 128 + q (bit pattern 0x4300 | q); X is split
// into a bf16 high part and a bf16 low part (two MFMAs per K step); per block
// y += c1 * P + c2 * S with S the block sum of the operand actually multiplied
// (hi + lo), obtained from the same A operands against a B of ones:
//   Q4_0:     w = d (q - 8)         -> c1 = d,    c2 = -136 d
//   Q4_K:     w = d sc q - dmin m   -> c1 = d sc, c2 = -(128 d sc + dmin m)
//
// X staging: each wave converts the X columns of its own K range, one step
// and one set of 4 tokens at a time, densely (every lane converts 8 values of
// one (token, block, quarter)), writes hi/lo to its private LDS slice, and
// reads them back in the block-diagonal arrangement (the 16 lanes with
// n/4 == g; the other lanes keep zero operands). Codes are decoded once per
// step for all token sets. Codes, scales and X are prefetched two steps ahead.
//
// Workgroup: NW waves on the same 16*RG rows, each on one contiguous range of
// K steps; the partials (over the four lane groups and the NW waves) are
// summed through LDS at the end.
#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

// names of the kernel templates, for lw_kernel_name
struct Name_multitok_kernel {
    static constexpr const char* base = "multitok_kernel";
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxWaves = 8;

// 16 code bytes of one block, read once (non-temporal).
__device__ __forceinline__ u32x4 load_codes(const uint8_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Code word j of a block -> the 8 bf16 values 128 + q of MFMA j: low nibbles
// (block elements 4j..4j+3), then high nibbles (16+4j..16+4j+3). v_perm_b32
// interleaves each code byte with a 0x43 byte: bf16 bits 0x4300 | q.
__device__ __forceinline__ bf16x8 biased_codes(uint32_t w) {
    const uint32_t lo = opaque(w & 0x0F0F0F0Fu);
    const uint32_t hi = opaque((w >> 4) & 0x0F0F0F0Fu);
    const uint32_t k43 = 0x43434343u;
    const u32x4 v = {__builtin_amdgcn_perm(k43, lo, 0x04010400u), __builtin_amdgcn_perm(k43, lo, 0x04030402u),
                     __builtin_amdgcn_perm(k43, hi, 0x04010400u), __builtin_amdgcn_perm(k43, hi, 0x04030402u)};
    return __builtin_bit_cast(bf16x8, v);
}

// Scale data of the lane's block, and its two coefficients.
template <int FMT>
struct Scale;

template <>
struct Scale<LW_Q4_0> {
    uint32_t h;  // binary16 d
    __device__ void load(const uint8_t* W, int64_t off1, int64_t, uint64_t row, uint32_t K, uint32_t blk) {
        h = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (row * (K / 32u) + blk));
    }
    __device__ void coef(uint32_t, float* c1, float* c2) const {
        const float d = half_bits_to_float(h);
        *c1 = d;
        *c2 = -136.0f * d;
    }
};

template <>
struct Scale<LW_Q4_K> {
    uint32_t a, b, c, dd;  // 96-bit scale record, {d, dmin}
    __device__ void load(const uint8_t* W, int64_t off1, int64_t off2, uint64_t row, uint32_t K, uint32_t blk) {
        const uint64_t sb = row * (K / 256u) + (blk >> 3);
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * sb);
        a = rec[0];
        b = rec[1];
        c = rec[2];
        dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * sb);
    }
    __device__ void coef(uint32_t blk, float* c1, float* c2) const {
        const uint32_t j = blk & 7u;
        const uint64_t lo = (uint64_t)a | ((uint64_t)b << 32);
        const uint64_t hi = (uint64_t)b | ((uint64_t)c << 32);
        const float ds = half_bits_to_float(dd & 0xFFFFu) * (float)((uint32_t)(lo >> (6 * j)) & 63u);
        const float dm = half_bits_to_float(dd >> 16) * (float)((uint32_t)(hi >> (16 + 6 * j)) & 63u);
        *c1 = ds;
        *c2 = -__builtin_fmaf(128.0f, ds, dm);
    }
};

template <int FMT, int NTS, int RG>
struct Stage {
    u32x4 codes[RG];
    Scale<FMT> sc[RG];
    float4 xa[NTS], xb[NTS];
};

template <int FMT, int NTS, int RG>
__global__ void __launch_bounds__(64 * kMaxWaves)
    multitok_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                    int64_t K, int ntok, int64_t off1, int64_t off2) {
    extern __shared__ float4 smem4[];
    const int nw = blockDim.x >> 6;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int n16 = lane & 15, g = lane >> 4;
    const uint32_t K32 = (uint32_t)K;

    // this wave's steps
    const int nsteps = (int)(K / 128);
    const int spw = (nsteps + nw - 1) / nw;
    const int s0 = wave * spw;
    const int s1 = (s0 + spw) < nsteps ? (s0 + spw) : nsteps;

    // rows of the lane in each row group (clamped; stores are masked)
    const int64_t row0 = (int64_t)blockIdx.x * 16 * RG;
    uint64_t row[RG];
    const uint8_t* cp[RG];
#pragma unroll
    for (int q = 0; q < RG; ++q) {
        const int64_t r = row0 + 16 * q + n16;
        row[q] = (uint64_t)(r < M ? r : M - 1);
        cp[q] = W + row[q] * (K32 / 2u) + 16u * g;
    }
    // dense X conversion: lane -> (quarter jd, block bd, token td of a token set)
    const int jd = lane >> 4, bd = (lane >> 2) & 3, td = lane & 3;
    const float* xp[NTS];
    bool xv[NTS];
#pragma unroll
    for (int ts = 0; ts < NTS; ++ts) {
        const int T = 4 * ts + td;
        xv[ts] = T < ntok;
        xp[ts] = x + (int64_t)(xv[ts] ? T : 0) * K + 32 * bd + 4 * jd;
    }
    // LDS: per wave, hi then lo of one token set, 64 x 16 bytes each
    float4* xs = smem4 + (size_t)wave * 128;
    const bool active = (n16 >> 2) == g;

    auto load = [&](Stage<FMT, NTS, RG>& st, int s) {
#pragma unroll
        for (int q = 0; q < RG; ++q) {
            st.codes[q] = load_codes(cp[q] + 64u * (uint32_t)s);
            st.sc[q].load(W, off1, off2, row[q], K32, 4u * (uint32_t)s + (uint32_t)g);
        }
#pragma unroll
        for (int ts = 0; ts < NTS; ++ts) {
            st.xa[ts] = *reinterpret_cast<const float4*>(xp[ts] + 128 * s);
            st.xb[ts] = *reinterpret_cast<const float4*>(xp[ts] + 128 * s + 16);
        }
    };

    const bf16x8 ones = __builtin_bit_cast(bf16x8, u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
    // block-diagonal A operands of one token set; the lanes outside the
    // diagonal never write them, so they stay zero
    bf16x8 ah[4], al[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        ah[j] = bf16x8{};
        al[j] = bf16x8{};
    }
    f32x4 acc[NTS][RG];
#pragma unroll
    for (int ts = 0; ts < NTS; ++ts)
#pragma unroll
        for (int q = 0; q < RG; ++q) acc[ts][q] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto consume = [&](const Stage<FMT, NTS, RG>& st, int s) {
        // codes of the step -> B operands, once for all token sets
        bf16x8 bq[RG][4];
#pragma unroll
        for (int q = 0; q < RG; ++q)
#pragma unroll
            for (int j = 0; j < 4; ++j) bq[q][j] = biased_codes(st.codes[q][j]);
        float c1[RG], c2[RG];
        const uint32_t blk = 4u * (uint32_t)s + (uint32_t)g;
#pragma unroll
        for (int q = 0; q < RG; ++q) st.sc[q].coef(blk, &c1[q], &c2[q]);
#pragma unroll
        for (int ts = 0; ts < NTS; ++ts) {
            // X of this step and token set: dense hi/lo conversion -> LDS ->
            // block-diagonal operands
            const float v[8] = {st.xa[ts].x, st.xa[ts].y, st.xa[ts].z, st.xa[ts].w,
                                st.xb[ts].x, st.xb[ts].y, st.xb[ts].z, st.xb[ts].w};
            bf16x8 h, l;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float ve = xv[ts] ? v[e] : 0.f;
                h[e] = (__bf16)ve;
                l[e] = (__bf16)(ve - (float)h[e]);
            }
            __builtin_amdgcn_wave_barrier();
            xs[lane] = __builtin_bit_cast(float4, h);
            xs[64 + lane] = __builtin_bit_cast(float4, l);
            __builtin_amdgcn_wave_barrier();
            if (active) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    ah[j] = __builtin_bit_cast(bf16x8, xs[16 * j + n16]);
                    al[j] = __builtin_bit_cast(bf16x8, xs[64 + 16 * j + n16]);
                }
            }
            __builtin_amdgcn_wave_barrier();
            // block sums of the multiplied operand (against ones), and the products
            f32x4 S = {0.f, 0.f, 0.f, 0.f};
            f32x4 P[RG];
#pragma unroll
            for (int q = 0; q < RG; ++q) P[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                S = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[j], ones, S, 0, 0, 0);
#pragma unroll
                for (int q = 0; q < RG; ++q) P[q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[j], bq[q][j], P[q], 0, 0, 0);
                S = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[j], ones, S, 0, 0, 0);
#pragma unroll
                for (int q = 0; q < RG; ++q) P[q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[j], bq[q][j], P[q], 0, 0, 0);
            }
#pragma unroll
            for (int q = 0; q < RG; ++q)
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4)
                    acc[ts][q][v4] = __builtin_fmaf(c2[q], S[v4], __builtin_fmaf(c1[q], P[q][v4], acc[ts][q][v4]));
        }
    };

    Stage<FMT, NTS, RG> sa, sb;
    if (s0 < s1) load(sa, s0);
    if (s0 + 1 < s1) load(sb, s0 + 1);
    for (int s = s0; s < s1; s += 2) {
        consume(sa, s);
        if (s + 2 < s1) load(sa, s + 2);
        if (s + 1 < s1) {
            consume(sb, s + 1);
            if (s + 3 < s1) load(sb, s + 3);
        }
    }

    // sum the partials over the 4 lane groups and the waves
    float* red = reinterpret_cast<float*>(smem4 + (size_t)nw * 128);  // [nw*4][NTS*4][16*RG]
    constexpr int kRows = 16 * RG, kTok = 4 * NTS;
#pragma unroll
    for (int ts = 0; ts < NTS; ++ts)
#pragma unroll
        for (int q = 0; q < RG; ++q)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                red[((wave * 4 + g) * kTok + 4 * ts + v) * kRows + 16 * q + n16] = acc[ts][q][v];
    __syncthreads();
    for (int it = tid; it < kTok * kRows; it += blockDim.x) {
        const int t = it / kRows, r = it % kRows;
        if (t < ntok && row0 + r < M) {
            float o = 0.f;
            for (int p = 0; p < nw * 4; ++p) o += red[(p * kTok + t) * kRows + r];
            y[(int64_t)t * M + row0 + r] = o;
        }
    }
}

template <int FMT, int NTS, int RG>
hipError_t launch3(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok, const Planes& p,
                   int nw, hipStream_t stream) {
    const int64_t grid = (M + 16 * RG - 1) / (16 * RG);
    if (grid > 0x7fffffff || nw < 1 || nw > kMaxWaves) return hipErrorInvalidConfiguration;
    const size_t lds = (size_t)nw * 128 * 16 + (size_t)nw * 4 * (4 * NTS) * (16 * RG) * 4;
    if (query_only(kernel_name<Name_multitok_kernel, FMT, NTS, RG>())) return hipSuccess;
    hipLaunchKernelGGL((multitok_kernel<FMT, NTS, RG>), dim3((unsigned)grid), dim3(64 * nw), lds, stream, W, x, y, M,
                       K, (int)n_tok, p.off1, p.off2);
    return hipGetLastError();
}

int cu_count_mt() {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
        return 256;
    return v;
}

template <int FMT>
hipError_t launch_f(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok, const Planes& p,
                    hipStream_t stream) {
    const int64_t cus = cu_count_mt();
    // two row groups per workgroup when that still leaves two workgroups per CU
    // (and registers allow: one row group for 13..16 tokens)
    const bool rg2 = (M + 31) / 32 >= 2 * cus && n_tok <= 12;
    const int64_t wgs = rg2 ? (M + 31) / 32 : (M + 15) / 16;
    const int nw = wgs >= 2 * cus ? 4 : 8;
    const int nts = (int)((n_tok + 3) / 4);
    if (rg2) {
        switch (nts) {
        case 1: return launch3<FMT, 1, 2>(W, x, y, M, K, n_tok, p, nw, stream);
        case 2: return launch3<FMT, 2, 2>(W, x, y, M, K, n_tok, p, nw, stream);
        case 3: return launch3<FMT, 3, 2>(W, x, y, M, K, n_tok, p, nw, stream);
        default: return hipErrorInvalidValue;
        }
    }
    switch (nts) {
    case 1: return launch3<FMT, 1, 1>(W, x, y, M, K, n_tok, p, nw, stream);
    case 2: return launch3<FMT, 2, 1>(W, x, y, M, K, n_tok, p, nw, stream);
    case 3: return launch3<FMT, 3, 1>(W, x, y, M, K, n_tok, p, nw, stream);
    case 4: return launch3<FMT, 4, 1>(W, x, y, M, K, n_tok, p, nw, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool multitok_supported(int fmt, int64_t n_tok) {
    return (fmt == LW_Q4_0 || fmt == LW_Q4_K) && n_tok >= 2 && n_tok <= 16;
}

hipError_t launch_multitok(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                           int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_f<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_f<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
