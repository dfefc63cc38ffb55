// Decode attention over a KV cache stored in a weight format.
//
// One query token (the decode step of Sec. 2.1) attends over kv_len cached
// positions; K and V are dequantized as they are loaded, with the same
// per-format routine as the weights (Sec. 3.2: attention reads quantized K
// and V; Sec. 3.3: the dequantization routines serve the KV cache). For
// query head h and its key/value head g = h / G (G = n_heads / n_kv_heads):
//   s_j = scale * q_h . k_{g,j},  p = softmax(s),  out_h = sum_j p_j v_{g,j}.
//
// Split over the positions (flash decoding): workgroup (g, s) takes the G
// query heads of key/value head g over positions [s*rps, (s+1)*rps) and
// writes per head the running maximum m, the sum l of exp(s_j - m) and the
// unnormalised output sum_j exp(s_j - m) v_j to the workspace; a second
// kernel rescales the splits to their common maximum and divides (scores and
// maxima are kept in base-2 units, s log2(e), so every exponential is one
// v_exp_f32 of a non-positive argument). Inside a
// workgroup each wave takes batches of RPW positions: lane (r, c) holds DPL
// consecutive dimensions c*DPL .. of position r, its query slices for the G
// heads in registers; scores are lane sums over the LPR = head_dim / DPL
// lanes of a position, and the online softmax rescales the lane's G x DPL
// output partials by exp(m_old - m_new) per batch. The wave's partials are
// then summed over positions by a reduce-scatter (two permlane swap steps,
// each halving the values a lane holds, then DPP row rotations), and the
// four waves combined through LDS. Everything is float32; every exp
// argument is <= 0.
#include <cmath>

#include "lw_device.hpp"
#include "lw_formats.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

struct Name_attn_split_kernel {
    static constexpr const char* base = "attn_split_kernel";
};

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;

template <int G>
constexpr int dims_per_lane() {
    return G <= 4 ? 16 : 8;
}

// Lane reductions without LDS round trips. partner<MASK> gives, for masks 1
// and 2, the DPP quad permutations (the lane's xor-MASK partner); for 4 and 8
// the DPP half-row and row mirrors (lane i with 7 - i, 15 - i), which stand
// in for the xor partner when the values are equal within groups of MASK
// lanes; for 16 and 32 the permlane swaps of rows and halves (exact xor
// partners).
template <int MASK>
__device__ __forceinline__ float partner(float v) {
    if constexpr (MASK == 1) return dpp_move<0xB1>(v);
    else if constexpr (MASK == 2) return dpp_move<0x4E>(v);
    else if constexpr (MASK == 4) return dpp_move<0x141>(v);
    else if constexpr (MASK == 8) return dpp_move<0x140>(v);
    else {
        const uint32_t b = __builtin_bit_cast(uint32_t, v);
        const auto sw = MASK == 16 ? __builtin_amdgcn_permlane16_swap(b, b, false, false)
                                   : __builtin_amdgcn_permlane32_swap(b, b, false, false);
        // the upper group of each pair finds its partner in the first result
        const int lane = threadIdx.x & (kWave - 1);
        return __builtin_bit_cast(float, (lane & MASK) ? sw[0] : sw[1]);
    }
}
// v summed (maximised) over the lanes that differ from this one in the mask
// bits LO .. HI - 1, for values already equal within aligned groups of LO
// lanes (LO a power of two; 1: no condition).
template <int LO, int HI>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr (LO < HI) return group_sum<2 * LO, HI>(v + partner<LO>(v));
    else return v;
}
template <int LO, int HI>
__device__ __forceinline__ float group_max(float v) {
    if constexpr (LO < HI) return group_max<2 * LO, HI>(fmaxf(v, partner<LO>(v)));
    else return v;
}
// v summed over all lanes congruent to this one modulo LO (LO = 4, 8 or 16),
// whatever the values: rotations of each 16-lane row by LO, 2 LO, ..., 8
// (DPP row_ror) reach every lane of the row in the same residue class, then
// the row and half swaps add the other rows.
template <int LO, int SH = LO>
__device__ __forceinline__ float residue_sum(float v) {
    if constexpr (SH < 16) return residue_sum<LO, 2 * SH>(v + dpp_move<0x120 + SH>(v));
    else return group_sum<16, kWave>(v);
}

// v summed over the lanes of its 16-lane row congruent to this one modulo LO
// (LO = 1 .. 16, a power of two; 16: v itself).
template <int LO, int SH = LO>
__device__ __forceinline__ float row_residue_sum(float v) {
    if constexpr (SH < 16) return row_residue_sum<LO, 2 * SH>(v + dpp_move<0x120 + SH>(v));
    else return v;
}

// Reduce-scatter of N per-lane values over the lanes that share this lane's
// value set apart from the row bits LO (a power of two, at most 16) .. 32 of
// the lane index: the halves of the set are exchanged across the 32-lane and
// the 16-lane halves with one permlane swap per two values (each lane then
// adds the half it keeps), and the row bits below 16 are summed with DPP row
// rotations. Afterwards out[j], j < N / 4, holds the total of value
// j + (N / 4) (bit 4) + (N / 2) (bit 5) of the lane index.
template <int N, int LO>
__device__ __forceinline__ void reduce_scatter(const float* v, float* out) {
    static_assert(N % 4 == 0 && LO >= 1 && LO <= 16, "whole quarters, row bits from LO");
    float w[N / 2];
#pragma unroll
    for (int j = 0; j < N / 2; ++j) {
        const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v[j]),
                                                        __builtin_bit_cast(uint32_t, v[j + N / 2]), false, false);
        uint32_t r0 = r[0], r1 = r[1];
        asm("" : "+v"(r0), "+v"(r1));  // else the compiler folds r[1] into r[0] when both are summed
        w[j] = __builtin_bit_cast(float, r0) + __builtin_bit_cast(float, r1);
    }
#pragma unroll
    for (int j = 0; j < N / 4; ++j) {
        const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, w[j]),
                                                        __builtin_bit_cast(uint32_t, w[j + N / 4]), false, false);
        uint32_t r0 = r[0], r1 = r[1];
        asm("" : "+v"(r0), "+v"(r1));  // else the compiler folds r[1] into r[0] when both are summed
        out[j] = __builtin_bit_cast(float, r0) + __builtin_bit_cast(float, r1);
    }
#pragma unroll
    for (int j = 0; j < N / 4; ++j) out[j] = row_residue_sum<LO>(out[j]);
}

template <int FMT, int D, int G>
__global__ void __launch_bounds__(kAttnThreads)
    attn_split_kernel(const float* __restrict__ q, const uint8_t* __restrict__ Kc, const uint8_t* __restrict__ Vc,
                      int64_t off1, int64_t off2, int64_t off3, int kv_len, int n_heads, float scale, int rps,
                      float* __restrict__ ws) {
    constexpr int DPL = dims_per_lane<G>();
    constexpr int LPR = D / DPL;       // lanes per position
    constexpr int RPW = kWave / LPR;   // positions per wave and batch
    __shared__ float red[kAttnWaves][G][D + 2];

    const int g = blockIdx.x, split = blockIdx.y;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int r = lane / LPR, c = lane - r * LPR;
    const int j0 = split * rps;
    // scores in base-2 units: exp(x) = exp2(x log2(e)), one v_exp_f32 each
    const float scale2 = scale * 1.4426950408889634f;
    const int j1 = min(kv_len, j0 + rps);

    float qv[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float4* qp = reinterpret_cast<const float4*>(q + (int64_t)(g * G + h) * D + c * DPL);
#pragma unroll
        for (int i = 0; i < DPL / 4; ++i) {
            const float4 t = qp[i];
            qv[h][4 * i] = t.x;
            qv[h][4 * i + 1] = t.y;
            qv[h][4 * i + 2] = t.z;
            qv[h][4 * i + 3] = t.w;
        }
    }
    float m[G], l[G], acc[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[h][i] = 0.f;
    }

    const int64_t head_base = (int64_t)g * kv_len;
    // one batch: positions b .. b + RPW - 1 (this lane: b + r), K and V decoded
    auto load_batch = [&](int b, float* kk, float* vv) __attribute__((always_inline)) {
        const int row = b + r;
        const int64_t e = (head_base + (row < j1 ? row : j1 - 1)) * D + c * DPL;
#pragma unroll
        for (int i = 0; i < DPL / 4; ++i) {
            const float4 t = value4<FMT>(Kc, off1, off2, off3, e + 4 * i);
            kk[4 * i] = t.x;
            kk[4 * i + 1] = t.y;
            kk[4 * i + 2] = t.z;
            kk[4 * i + 3] = t.w;
        }
#pragma unroll
        for (int i = 0; i < DPL / 4; ++i) {
            const float4 t = value4<FMT>(Vc, off1, off2, off3, e + 4 * i);
            vv[4 * i] = t.x;
            vv[4 * i + 1] = t.y;
            vv[4 * i + 2] = t.z;
            vv[4 * i + 3] = t.w;
        }
    };
    auto consume = [&](int b, const float* kk, const float* vv) __attribute__((always_inline)) {
        const bool valid = b + r < j1;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float d = 0.f;
#pragma unroll
            for (int i = 0; i < DPL; ++i) d = __builtin_fmaf(qv[h][i], kk[i], d);
            d = group_sum<1, LPR>(d);
            const float s = valid ? d * scale2 : -INFINITY;
            const float mb = group_max<LPR, kWave>(s);
            const float mn = fmaxf(m[h], mb);  // finite: the batch has a valid position
            if (mn != m[h]) {                  // wave-uniform: a new maximum rescales the partials
                const float alpha = __builtin_amdgcn_exp2f(m[h] - mn);  // m = -inf: 0
                m[h] = mn;
                l[h] *= alpha;
#pragma unroll
                for (int i = 0; i < DPL; ++i) acc[h][i] *= alpha;
            }
            const float p = valid ? __builtin_amdgcn_exp2f(s - mn) : 0.f;
            l[h] += c == 0 ? p : 0.f;
#pragma unroll
            for (int i = 0; i < DPL; ++i) acc[h][i] = __builtin_fmaf(p, vv[i], acc[h][i]);
        }
    };
    // two batches per round, both loaded before either is used (twice the
    // bytes in flight per wave); the second only where it starts inside
    // the split
    constexpr int kStep = kAttnWaves * RPW;
    for (int b = j0 + wave * RPW; b < j1; b += 2 * kStep) {
        float k0[DPL], v0[DPL], k1[DPL], v1[DPL];
        const bool two = b + kStep < j1;
        load_batch(b, k0, v0);
        load_batch(two ? b + kStep : b, k1, v1);
        consume(b, k0, v0);
        if (two) consume(b + kStep, k1, v1);
    }

    // the wave's totals: l over all lanes, the outputs over the positions
    // (the G * DPL sums over the wave's positions: a reduce-scatter leaves a
    // quarter of them in each lane, which the first LPR lanes of each
    // 16-lane row store)
    {
        constexpr int N = G * DPL;
        float v[N], tot[N / 4];
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int i = 0; i < DPL; ++i) v[h * DPL + i] = acc[h][i];
        reduce_scatter<N, LPR>(v, tot);
        const int J0 = ((lane >> 4) & 1) * (N / 4) + ((lane >> 5) & 1) * (N / 2);
        if ((lane & 15) < LPR) {
#pragma unroll
            for (int j = 0; j < N / 4; ++j) {
                const int J = J0 + j;
                red[wave][J / DPL][c * DPL + J % DPL] = tot[j];
            }
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float lt = group_sum<1, kWave>(l[h]);
        if (lane == 0) {
            red[wave][h][D] = m[h];
            red[wave][h][D + 1] = lt;
        }
    }
    __syncthreads();
    // combine the waves (a wave without positions has m = -inf, l = 0, sums 0)
    float* out = ws + ((int64_t)split * n_heads + (int64_t)g * G) * (D + 2);
    for (int idx = threadIdx.x; idx < G * (D + 2); idx += kAttnThreads) {
        const int h = idx / (D + 2), d = idx - h * (D + 2);
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, red[w][h][D]);
        float v = 0.f;
        if (d == D) {
            v = M;
        } else {
#pragma unroll
            for (int w = 0; w < kAttnWaves; ++w) {
                const float mw = red[w][h][D];
                const float wgt = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - M);
                v = __builtin_fmaf(wgt, red[w][h][d], v);
            }
        }
        out[(int64_t)h * (D + 2) + d] = v;
    }
}

// out[h][d] = sum_s exp(m_s - M) acc_s[d] / sum_s exp(m_s - M) l_s. One
// workgroup per head: every thread loads the maxima of its splits at once
// (one round trip for all of them), the weights w_s = exp(m_s - M) go to
// LDS, then thread (d, sg) sums the splits sg, sg + SG, ... of output d
// with sixteen loads in flight, and the SG partials are added through LDS.
constexpr int kCombThreads = 256;
constexpr int kMaxSplits = 1024;

template <int D>
__global__ void __launch_bounds__(kCombThreads) attn_combine_kernel(const float* __restrict__ ws,
                                                                   float* __restrict__ out, int n_heads, int splits) {
    constexpr int SG = kCombThreads / D;  // split groups
    __shared__ float wsp[kMaxSplits];
    __shared__ float part[SG][D + 1];
    __shared__ float red[kCombThreads / kWave];
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* base = ws + (int64_t)h * (D + 2);
    const int64_t stride = (int64_t)n_heads * (D + 2);
    // maxima of the splits: all loads first, then the reduction
    float mloc[kMaxSplits / kCombThreads];
#pragma unroll
    for (int i = 0; i < kMaxSplits / kCombThreads; ++i) {
        const int s = tid + i * kCombThreads;
        mloc[i] = s < splits ? base[s * stride + D] : -INFINITY;
    }
    float M = -INFINITY;
#pragma unroll
    for (int i = 0; i < kMaxSplits / kCombThreads; ++i) M = fmaxf(M, mloc[i]);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) M = fmaxf(M, __shfl_xor(M, o, kWave));
    if ((tid & (kWave - 1)) == 0) red[tid / kWave] = M;
    __syncthreads();
    M = red[0];
#pragma unroll
    for (int w = 1; w < kCombThreads / kWave; ++w) M = fmaxf(M, red[w]);
#pragma unroll
    for (int i = 0; i < kMaxSplits / kCombThreads; ++i) {
        const int s = tid + i * kCombThreads;
        if (s < splits) wsp[s] = mloc[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mloc[i] - M);
    }
    __syncthreads();
    // thread (d, sg) sums output d over the splits sg, sg + SG, ...; thread
    // d = 1 also sums l (slot D + 1) in the same pass. Sixteen splits' loads
    // (thirty-two for d = 1) are issued before any is used.
    const int sg = tid / D, d0 = tid - sg * D;
    const bool with_l = d0 == 1;
    constexpr int U = 16;
    float o = 0.f, ol = 0.f;
    int s = sg;
    for (; s + (U - 1) * SG < splits; s += U * SG) {
        float v[U], vl[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            v[u] = base[(s + u * SG) * stride + d0];
            vl[u] = with_l ? base[(s + u * SG) * stride + D + 1] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            o = __builtin_fmaf(wsp[s + u * SG], v[u], o);
            ol = __builtin_fmaf(wsp[s + u * SG], vl[u], ol);
        }
    }
    for (; s < splits; s += SG) {
        o = __builtin_fmaf(wsp[s], base[s * stride + d0], o);
        if (with_l) ol = __builtin_fmaf(wsp[s], base[s * stride + D + 1], ol);
    }
    part[sg][d0] = o;
    if (with_l) part[sg][D] = ol;
    __syncthreads();
    if (tid < D) {
        float o = 0.f, L = 0.f;
#pragma unroll
        for (int g = 0; g < SG; ++g) {
            o += part[g][tid];
            L += part[g][D];
        }
        out[(int64_t)h * D + tid] = o / L;
    }
}

template <int FMT, int D, int G>
hipError_t launch_g(const float* q, const uint8_t* K, const uint8_t* V, float* out, int64_t n_heads, int64_t n_kv,
                    int64_t kv_len, float scale, const AttnPlan& pl, float* ws, hipStream_t stream) {
    const Planes p = planes_of(FMT, n_kv * kv_len * D);
    if (query_only(kernel_name<Name_attn_split_kernel, FMT, D, G>(), 2)) return hipSuccess;
    hipLaunchKernelGGL((attn_split_kernel<FMT, D, G>), dim3((unsigned)n_kv, (unsigned)pl.splits), dim3(kAttnThreads),
                       0, stream, q, K, V, p.off1, p.off2, p.off3, (int)kv_len, (int)n_heads, scale, (int)pl.rps, ws);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((attn_combine_kernel<D>), dim3((unsigned)n_heads), dim3(kCombThreads), 0, stream, ws, out,
                       (int)n_heads, (int)pl.splits);
    return hipGetLastError();
}

template <int FMT, int D>
hipError_t launch_d(const float* q, const uint8_t* K, const uint8_t* V, float* out, int64_t n_heads, int64_t n_kv,
                    int64_t kv_len, float scale, const AttnPlan& pl, float* ws, hipStream_t stream) {
    switch (n_heads / n_kv) {
    case 1: return launch_g<FMT, D, 1>(q, K, V, out, n_heads, n_kv, kv_len, scale, pl, ws, stream);
    case 2: return launch_g<FMT, D, 2>(q, K, V, out, n_heads, n_kv, kv_len, scale, pl, ws, stream);
    case 4: return launch_g<FMT, D, 4>(q, K, V, out, n_heads, n_kv, kv_len, scale, pl, ws, stream);
    case 8: return launch_g<FMT, D, 8>(q, K, V, out, n_heads, n_kv, kv_len, scale, pl, ws, stream);
    default: return hipErrorInvalidValue;
    }
}

template <int FMT>
hipError_t launch_f(const float* q, const uint8_t* K, const uint8_t* V, float* out, int64_t n_heads, int64_t n_kv,
                    int64_t head_dim, int64_t kv_len, float scale, const AttnPlan& pl, float* ws,
                    hipStream_t stream) {
    if (head_dim == 64) return launch_d<FMT, 64>(q, K, V, out, n_heads, n_kv, kv_len, scale, pl, ws, stream);
    if (head_dim == 128) return launch_d<FMT, 128>(q, K, V, out, n_heads, n_kv, kv_len, scale, pl, ws, stream);
    return hipErrorInvalidValue;
}

}  // namespace

AttnPlan attn_plan(int64_t n_kv, int64_t head_dim, int64_t kv_len, int64_t n_heads) {
    AttnPlan pl;
    // about two workgroups per compute unit, at least 64 positions each (two
    // batches per wave: the per-wave reductions are paid once per split)
    const int64_t by_len = (kv_len + 63) / 64;
    const int64_t by_chip = (512 + n_kv - 1) / n_kv;
    int64_t splits = by_len < by_chip ? by_len : by_chip;
    if (splits < 1) splits = 1;
    pl.rps = (kv_len + splits - 1) / splits;
    pl.splits = (kv_len + pl.rps - 1) / pl.rps;  // no empty split
    pl.ws_bytes = pl.splits * n_heads * (head_dim + 2) * 4;
    return pl;
}

bool attn_fmt_supported(int fmt) {
    return fmt == LW_F16 || fmt == LW_Q8_0 || fmt == LW_Q4_0 || fmt == LW_Q4_1 || fmt == LW_Q5_0 || fmt == LW_Q5_1 ||
           fmt == LW_MXFP4;
}

hipError_t launch_attn(int fmt, const float* q, const uint8_t* K, const uint8_t* V, float* out, int64_t n_heads,
                       int64_t n_kv, int64_t head_dim, int64_t kv_len, float scale, const AttnPlan& pl, float* ws,
                       hipStream_t stream) {
    switch (fmt) {
    case LW_F16: return launch_f<LW_F16>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    case LW_Q8_0: return launch_f<LW_Q8_0>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    case LW_Q4_0: return launch_f<LW_Q4_0>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    case LW_Q4_1: return launch_f<LW_Q4_1>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    case LW_Q5_0: return launch_f<LW_Q5_0>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    case LW_Q5_1: return launch_f<LW_Q5_1>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    case LW_MXFP4: return launch_f<LW_MXFP4>(q, K, V, out, n_heads, n_kv, head_dim, kv_len, scale, pl, ws, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
