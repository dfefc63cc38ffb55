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
// lanes of a position. Batches come in sets of NB, two sets in flight per
// wave: the next set's loads are issued before the current set is decoded
// (f16, Q8_0 and Q4_0 keep the raw words until then; Q8_0 and Q4_0 decode
// to exact signed codes, the block scale applied once per head to the
// score and the weight instead of once per element). The online
// softmax takes one maximum per head over the whole set and rescales the
// lane's G x DPL output partials by exp(m_old - m_new) only when a maximum
// grew. The wave's partials are then summed over positions by a
// reduce-scatter (two permlane swap steps, each halving the values a lane
// holds, then DPP row rotations), and the four waves combined through LDS.
// Everything is float32; every exp argument is <= 0.
//
// f16, Q8_0 and Q4_0 caches whose splits hold more than 64 positions take
// attn_mf_kernel instead: the same split, online softmax and output
// accumulation, with the scores of 16-position tiles on the matrix cores
// (f16 operands: exact forms of the cache elements and the query as two f16
// parts; its header below states the exactness argument).
#include <cmath>

#include "lw_device.hpp"
#include "lw_formats.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

struct Name_attn_split_kernel {
    static constexpr const char* base = "attn_split_kernel";
};
struct Name_attn_mf_kernel {
    static constexpr const char* base = "attn_mf_kernel";
};

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;
// batches per set of the vector kernel's raw K/V loads (f16, Q8_0, Q4_0):
// four would take more than 256 registers with four heads per KV head
constexpr int kAttnRawBatches = 2;
// positions per split above which f16, Q8_0 and Q4_0 take the matrix-core
// score kernel (one round of 64 positions: the vector kernel)
constexpr int64_t kMfMinRps = 64;

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

// Raw K/V loads for f16, Q8_0 and Q4_0: the lane's DPL elements of a row
// (consecutive, inside one 32-element block) are kept as loaded, a few
// words per row, and decoded only when the batch is used, so that further
// batches stay in flight meanwhile. Q8_0 and Q4_0 decode to the signed
// integer codes c_i (Q8_0: one v_cvt_f32_i32 of a sign-extended byte; Q4_0:
// the nibble minus 8), exact, with value a * c_i for the block scale a = d,
// so the scale multiplies once per lane and head instead of once per element.
// A code of zero stays an exact zero: a cache dimension whose values are all
// zero gives an output of exactly zero, as the accuracy bound requires.
template <int FMT, int DPL>
struct AttnRaw {
    static constexpr bool kOn = FMT == LW_F16 || FMT == LW_Q8_0 || FMT == LW_Q4_0;
    static constexpr bool kAffine = FMT == LW_Q8_0 || FMT == LW_Q4_0;
    static constexpr int kWords = FMT == LW_F16 ? DPL / 2 : DPL / 4;
    // the other formats: the values, decoded by the element routine on load
    struct Raw {
        uint32_t w[kOn ? kWords : DPL];
        uint32_t s;
    };
    // element e of the plane (e a multiple of DPL)
    __device__ static void load(const uint8_t* __restrict__ P, int64_t off1, int64_t off2, int64_t off3, int64_t e,
                                Raw& x) {
        if constexpr (kOn) {
            // Q4_0: block e / 32 holds element 32g + i in the low nibble of
            // byte i and 32g + i + 16 in the high nibble of the same byte
            const uint8_t* p = FMT == LW_F16 ? P + 2 * e : FMT == LW_Q8_0 ? P + e : P + 16 * (e >> 5) + (e & 15);
#pragma unroll
            for (int k = 0; k < kWords; k += 4) {
                if constexpr (kWords >= 4) {
                    const uint4 t = *reinterpret_cast<const uint4*>(p + 4 * k);
                    x.w[k] = t.x;
                    x.w[k + 1] = t.y;
                    x.w[k + 2] = t.z;
                    x.w[k + 3] = t.w;
                } else {
                    const uint2 t = *reinterpret_cast<const uint2*>(p);
                    x.w[0] = t.x;
                    x.w[1] = t.y;
                }
            }
            if constexpr (kAffine) x.s = *reinterpret_cast<const uint16_t*>(P + off1 + 2 * (e >> 5));
        } else {
#pragma unroll
            for (int i = 0; i < DPL / 4; ++i) {
                const float4 t = value4<FMT>(P, off1, off2, off3, e + 4 * i);
                x.w[4 * i] = __builtin_bit_cast(uint32_t, t.x);
                x.w[4 * i + 1] = __builtin_bit_cast(uint32_t, t.y);
                x.w[4 * i + 2] = __builtin_bit_cast(uint32_t, t.z);
                x.w[4 * i + 3] = __builtin_bit_cast(uint32_t, t.w);
            }
        }
    }
    // the same from the lane's code bytes cp and its block's scale sp
    // (f16, Q8_0, Q4_0)
    __device__ static void load_ptr(const uint8_t* __restrict__ cp, const uint8_t* __restrict__ sp, Raw& x) {
        static_assert(kOn, "raw formats");
#pragma unroll
        for (int k = 0; k < kWords; k += 4) {
            if constexpr (kWords >= 4) {
                const uint4 t = *reinterpret_cast<const uint4*>(cp + 4 * k);
                x.w[k] = t.x;
                x.w[k + 1] = t.y;
                x.w[k + 2] = t.z;
                x.w[k + 3] = t.w;
            } else {
                const uint2 t = *reinterpret_cast<const uint2*>(cp);
                x.w[0] = t.x;
                x.w[1] = t.y;
            }
        }
        if constexpr (kAffine) x.s = *reinterpret_cast<const uint16_t*>(sp);
    }
    // sh: the Q4_0 nibble (0 or 4), the same for every row of a lane
    __device__ static void decode(const Raw& x, int sh, float* c, float& a) {
        a = 1.f;
        if constexpr (FMT == LW_F16) {
#pragma unroll
            for (int k = 0; k < kWords; ++k) {
                c[2 * k] = half_bits_to_float(x.w[k] & 0xFFFFu);
                c[2 * k + 1] = half_bits_to_float(x.w[k] >> 16);
            }
        } else if constexpr (kAffine) {
#pragma unroll
            for (int k = 0; k < kWords; ++k) {
                if constexpr (FMT == LW_Q8_0) {
                    c[4 * k] = sbyte<0>(x.w[k]);
                    c[4 * k + 1] = sbyte<1>(x.w[k]);
                    c[4 * k + 2] = sbyte<2>(x.w[k]);
                    c[4 * k + 3] = sbyte<3>(x.w[k]);
                } else {
                    const uint32_t w = opaque((x.w[k] >> sh) & 0x0F0F0F0Fu);
                    c[4 * k] = ubyte<0>(w) - 8.0f;
                    c[4 * k + 1] = ubyte<1>(w) - 8.0f;
                    c[4 * k + 2] = ubyte<2>(w) - 8.0f;
                    c[4 * k + 3] = ubyte<3>(w) - 8.0f;
                }
            }
            a = half_bits_to_float(x.s);
        } else {
#pragma unroll
            for (int i = 0; i < DPL; ++i) c[i] = __builtin_bit_cast(float, x.w[i]);
        }
    }
};

// The G x DPL output partials of a wave (lane (r, c): position r, dimensions
// c*DPL ..), summed over the wave's positions into row[h][0 .. D): a
// reduce-scatter leaves a quarter of the sums in each lane, which the first
// LPR lanes of each 16-lane row store.
template <int D, int G, int DPL>
__device__ __forceinline__ void wave_outputs_to_lds(const float* v, float (*row)[D + 2], int lane, int c) {
    constexpr int N = G * DPL, LPR = D / DPL;
    float tot[N / 4];
    reduce_scatter<N, LPR>(v, tot);
    const int J0 = ((lane >> 4) & 1) * (N / 4) + ((lane >> 5) & 1) * (N / 2);
    if ((lane & 15) < LPR) {
#pragma unroll
        for (int j = 0; j < N / 4; ++j) {
            const int J = J0 + j;
            row[J / DPL][c * DPL + J % DPL] = tot[j];
        }
    }
}

// The workgroup's waves merged (red[w][h]: outputs, then m and l; a wave
// without positions has m = -inf, l = 0, outputs 0) into the split's
// workspace record out[h][0 .. D + 2).
template <int D, int G>
__device__ __forceinline__ void merge_waves(float (*red)[G][D + 2], float* __restrict__ out) {
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
    // wave-uniform in a scalar register: the loop over the sets below
    // then branches on scalars, and its waits can leave loads in flight
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
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
    using RW = AttnRaw<FMT, DPL>;
    constexpr bool kAff = RW::kAffine;
    float m[G], l[G], acc[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[h][i] = 0.f;
    }

    const int64_t head_base = (int64_t)g * kv_len;
    // a batch: positions b .. b + RPW - 1 (this lane: b + r; rows past the
    // split repeat its last row and are masked)
    constexpr int kStep = kAttnWaves * RPW;
    auto elem = [&](int b) __attribute__((always_inline)) {
        const int row = b + r;
        return (head_base + (row < j1 ? row : j1 - 1)) * D + c * DPL;
    };
    // a set: NB batches b, b + kStep, ... loaded together. K and V of f16,
    // Q8_0 and Q4_0 stay as loaded until the set is used; the other formats
    // are decoded on load (their values take more registers: one batch)
    constexpr int NB = RW::kOn ? kAttnRawBatches : 1;
    using Raw = typename RW::Raw;
    const int sh = (c * DPL) & 16 ? 4 : 0;
    auto load_set = [&](int b, Raw* kr, Raw* vr) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int64_t e = elem(b + i * kStep);
            RW::load(Kc, off1, off2, off3, e, kr[i]);
            RW::load(Vc, off1, off2, off3, e, vr[i]);
        }
    };
    // the set's scores for every head, then one maximum per head over the
    // set (one rescale test per set, no branch between the heads), then
    // the weights and the output partials
    auto use_set = [&](int b, const Raw* kr, const Raw* vr) __attribute__((always_inline)) {
        float s[NB][G];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            float kk[DPL], ka;
            RW::decode(kr[i], sh, kk, ka);
            const bool valid = b + i * kStep + r < j1;
#pragma unroll
            for (int h = 0; h < G; ++h) {
                float d = 0.f;
#pragma unroll
                for (int k = 0; k < DPL; ++k) d = __builtin_fmaf(qv[h][k], kk[k], d);
                if constexpr (kAff) d *= ka;
                d = group_sum<1, LPR>(d);
                s[i][h] = valid ? d * scale2 : -INFINITY;
            }
        }
        float mn[G];
        bool grow = false;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float mb = s[0][h];
#pragma unroll
            for (int i = 1; i < NB; ++i) mb = fmaxf(mb, s[i][h]);
            mb = group_max<LPR, kWave>(mb);
            mn[h] = fmaxf(m[h], mb);  // finite: the first set has a valid position
            grow |= mn[h] != m[h];
        }
        if (__builtin_amdgcn_readfirstlane((int)grow)) {  // wave-uniform: a new maximum rescales the partials
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float alpha = __builtin_amdgcn_exp2f(m[h] - mn[h]);  // m = -inf: 0; unchanged: 1
                m[h] = mn[h];
                l[h] *= alpha;
#pragma unroll
                for (int k = 0; k < DPL; ++k) acc[h][k] *= alpha;
            }
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            float vv[DPL], va;
            RW::decode(vr[i], sh, vv, va);
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float p = __builtin_amdgcn_exp2f(s[i][h] - m[h]);  // masked (s = -inf): 0
                l[h] += p;  // in all LPR lanes of the position: LPR times the sum
                const float pa = kAff ? p * va : p;
#pragma unroll
                for (int k = 0; k < DPL; ++k) acc[h][k] = __builtin_fmaf(pa, vv[k], acc[h][k]);
            }
        }
    };
    // two sets alternate: the next is issued before the current one is
    // used, so a set per wave is in flight while it computes (unrolled by
    // hand over the two: no register copies of data still in flight). The
    // next set is loaded unconditionally (past the split: its last row
    // again, from the cache), and the loop has one exit and a wave-uniform
    // trip count, so that every wait for the current set can leave the
    // next one's loads outstanding.
    int b = j0 + wave * RPW;
    if (b < j1) {
        constexpr int kSet = NB * kStep;
        const int n = (j1 - b + kSet - 1) / kSet;  // the wave's sets
        Raw ka[NB], va[NB], kb[NB], vb[NB];
        load_set(b, ka, va);
        for (int t = 2; t <= n; t += 2) {
            load_set(b + kSet, kb, vb);
            use_set(b, ka, va);
            load_set(b + 2 * kSet, ka, va);
            use_set(b + kSet, kb, vb);
            b += 2 * kSet;
        }
        if (n & 1) use_set(b, ka, va);
    }

    // the wave's totals: l over all lanes, the outputs over the positions
    {
        float v[G * DPL];
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int i = 0; i < DPL; ++i) v[h * DPL + i] = acc[h][i];
        wave_outputs_to_lds<D, G, DPL>(v, red[wave], lane, c);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
        // each position's weight counted once per lane of the position:
        // LPR (a power of 2) times the sum, the scaling exact
        const float lt = group_sum<1, kWave>(l[h]) * (1.0f / LPR);
        if (lane == 0) {
            red[wave][h][D] = m[h];
            red[wave][h][D + 1] = lt;
        }
    }
    __syncthreads();
    merge_waves<D, G>(red, ws + ((int64_t)split * n_heads + (int64_t)g * G) * (D + 2));
}

// Scores on the matrix cores (f16, Q8_0 and Q4_0 caches). A wave takes
// tiles of 16 positions; v_mfma_f32_16x16x32_f16 multiplies the tile's K
// rows (A: row n = position n of the tile, one 32-element block per
// instruction) by the query (B: column n < G the high f16 part of head n,
// column G + n its low part, the other columns zero), so lane (gq, n)
// receives column n of rows 4gq .. 4gq + 3. Each lane group gq supplies 8
// elements of every block: f16 and Q8_0 elements 8gq .. 8gq + 7, Q4_0 the low
// and then the high nibbles of bytes 4gq .. 4gq + 3 (elements 4gq .. and
// 16 + 4gq ..); the query columns follow the same order.
//
// Exactness. Q8_0 codes enter as the f16 1024 + (q + 128) (bits 0x64 and the
// code with its sign bit flipped, one v_perm per two codes), Q4_0 nibbles as
// 1024 + c: the accumulator starts at -1152 (Q8_0) or -1032 (Q4_0) times the
// block's sum of the query part, so it ends at the sum of the query part
// times the signed code, and the block scale multiplies it afterwards. The
// query is first scaled by a power of two per head (its largest magnitude
// into [2^13, 2^14), so no f16 part overflows) and split into high and low
// f16 parts, 22 significant bits; products are exact in the float32
// accumulation and the scaling is undone exactly with the score scale.
// The weights p then go through LDS to the value layout of the vector path
// (lane (r, c): position r, dimensions c*DPL ..), which accumulates the
// outputs as the split kernel does.
template <int FMT, int D, int G>
__global__ void __launch_bounds__(kAttnThreads)
    attn_mf_kernel(const float* __restrict__ q, const uint8_t* __restrict__ Kc, const uint8_t* __restrict__ Vc,
                   int64_t off1, int kv_len, int n_heads, float scale, int rps, float* __restrict__ ws) {
    typedef _Float16 h16x8 __attribute__((ext_vector_type(8)));
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    static_assert(FMT == LW_F16 || FMT == LW_Q8_0 || FMT == LW_Q4_0, "f16, Q8_0 and Q4_0 caches");
    static_assert(2 * G <= 16, "high and low parts of every head in 16 columns");
    constexpr int NBK = D / 32;                          // blocks per row
    constexpr int DPL = dims_per_lane<G>();
    constexpr int LPR = D / DPL;                          // value layout: lanes per position
    constexpr int RPW = kWave / LPR;                      // positions per value batch
    constexpr int BPT = 16 / RPW;                         // value batches per tile
    constexpr int KW = FMT == LW_F16 ? 4 : FMT == LW_Q8_0 ? 2 : 1;  // K words per block and lane
    constexpr int SW = NBK / 2;                           // scale words per row (two f16 each)
    constexpr bool kScaled = FMT != LW_F16;
    constexpr float kBias = FMT == LW_Q8_0 ? 1152.0f : 1032.0f;
    using RW = AttnRaw<FMT, DPL>;
    using Raw = typename RW::Raw;
    __shared__ float red[kAttnWaves][G][D + 2];
    __shared__ float pw[kAttnWaves][16][G];              // the tile's weights [position][head]

    const int g = blockIdx.x, split = blockIdx.y;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int n = lane & 15, gq = lane >> 4;             // score layout
    const int r = lane / LPR, c = lane - r * LPR;        // value layout
    const int j0 = split * rps;
    const int j1 = min(kv_len, j0 + rps);
    const int64_t head_base = (int64_t)g * kv_len;

    // the query operand, its per-head power-of-two scaling, the bias sums
    h16x8 bq[NBK];
    float cb[NBK];
    float sc;  // column n < G: the score factor scale * log2(e) * 2^-shift
    {
        const bool qcol = n < 2 * G;
        const int hq = n < G ? n : n - G;
        const float* qh = q + (int64_t)(g * G + (qcol ? hq : 0)) * D;
        float qf[NBK][8];
#pragma unroll
        for (int bk = 0; bk < NBK; ++bk) {
            const int d0 = 32 * bk + (FMT == LW_Q4_0 ? 4 * gq : 8 * gq);
            const float4 a = *reinterpret_cast<const float4*>(qh + d0);
            const float4 b = *reinterpret_cast<const float4*>(qh + d0 + (FMT == LW_Q4_0 ? 16 : 4));
            qf[bk][0] = a.x;
            qf[bk][1] = a.y;
            qf[bk][2] = a.z;
            qf[bk][3] = a.w;
            qf[bk][4] = b.x;
            qf[bk][5] = b.y;
            qf[bk][6] = b.z;
            qf[bk][7] = b.w;
        }
        float amax = 0.f;
#pragma unroll
        for (int bk = 0; bk < NBK; ++bk)
#pragma unroll
            for (int k = 0; k < 8; ++k) amax = fmaxf(amax, fabsf(qf[bk][k]));
        amax = fmaxf(amax, partner<16>(amax));
        amax = fmaxf(amax, partner<32>(amax));  // the head's largest magnitude, in its four lane groups
        int ex;
        (void)frexpf(amax, &ex);  // amax < 2^ex (amax = 0: ex = 0)
        const int shift = 14 - ex;
        sc = scale * 1.4426950408889634f * ldexpf(1.0f, -shift);
#pragma unroll
        for (int bk = 0; bk < NBK; ++bk) {
            float part = 0.f;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const float qs = ldexpf(qf[bk][k], shift);  // exact
                const _Float16 hi = (_Float16)qs;
                const _Float16 lo = (_Float16)(qs - (float)hi);
                const _Float16 v = !qcol ? (_Float16)0.0f : n < G ? hi : lo;
                bq[bk][k] = v;
                part += (float)v;
            }
            part += partner<16>(part);
            part += partner<32>(part);  // the block's sum of this column's part
            cb[bk] = kScaled ? -kBias * part : 0.f;
        }
    }

    float m_l = -INFINITY, l_l = 0.f;  // lane (gq, n < G): head n's running maximum; its rows' weight sum
    float acc[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[h][i] = 0.f;
    const int sh = (c * DPL) & 16 ? 4 : 0;

    struct Tile {
        uint32_t kw[NBK][KW];     // K: the lane's row, its 8 elements of each block
        uint32_t ks[4][SW];       // K scales of rows 4gq .. 4gq + 3
        Raw v[BPT];               // V in the value layout
    };
    // per-row byte strides of the code and scale planes, and the lane's
    // base addresses in this head's rows (row j at base + j * stride)
    constexpr uint32_t kRowB = FMT == LW_F16 ? 2 * D : FMT == LW_Q8_0 ? D : D / 2;
    constexpr uint32_t kRowS = 2 * NBK;
    const uint8_t* kbase = Kc + head_base * kRowB +
                           (FMT == LW_F16 ? 16 * gq : FMT == LW_Q8_0 ? 8 * gq : 4 * gq);
    const uint8_t* ksbase = Kc + off1 + head_base * kRowS;
    const int ce = c * DPL;  // the lane's first dimension in the value layout
    const uint8_t* vbase = Vc + head_base * kRowB +
                           (FMT == LW_F16 ? 2 * ce : FMT == LW_Q8_0 ? ce : 16 * (ce >> 5) + (ce & 15));
    const uint8_t* vsbase = Vc + off1 + head_base * kRowS + 2 * (ce >> 5);
    const uint32_t jl = (uint32_t)(j1 - 1);
    auto clamp = [&](int row) __attribute__((always_inline)) {
        return (uint64_t)min((uint32_t)row, jl);
    };
    // a tile: positions b .. b + 15 (rows past the split repeat its last row
    // and are masked)
    auto load_tile = [&](int b, Tile& t) __attribute__((always_inline)) {
        const uint8_t* kp = kbase + clamp(b + n) * kRowB;
#pragma unroll
        for (int bk = 0; bk < NBK; ++bk) {
            if constexpr (FMT == LW_F16) {
                const uint4 w = *reinterpret_cast<const uint4*>(kp + 64 * bk);
                t.kw[bk][0] = w.x;
                t.kw[bk][1] = w.y;
                t.kw[bk][2] = w.z;
                t.kw[bk][3] = w.w;
            } else if constexpr (FMT == LW_Q8_0) {
                const uint2 w = *reinterpret_cast<const uint2*>(kp + 32 * bk);
                t.kw[bk][0] = w.x;
                t.kw[bk][1] = w.y;
            } else {
                t.kw[bk][0] = *reinterpret_cast<const uint32_t*>(kp + 16 * bk);
            }
        }
        if constexpr (kScaled) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint8_t* sp = ksbase + clamp(b + 4 * gq + i) * kRowS;
                if constexpr (SW == 2) {
                    const uint2 w = *reinterpret_cast<const uint2*>(sp);
                    t.ks[i][0] = w.x;
                    t.ks[i][1] = w.y;
                } else {
                    t.ks[i][0] = *reinterpret_cast<const uint32_t*>(sp);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < BPT; ++j) {
            const uint64_t row = clamp(b + j * RPW + r);
            RW::load_ptr(vbase + row * kRowB, vsbase + row * kRowS, t.v[j]);
        }
    };
    auto use_tile = [&](int b, const Tile& t) __attribute__((always_inline)) {
        // scores of rows 4gq + i, column n
        float S[4];
        if constexpr (FMT == LW_F16) {
            f32x4 C = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int bk = 0; bk < NBK; ++bk) {
                const uint32_t w[4] = {t.kw[bk][0], t.kw[bk][1], t.kw[bk][2], t.kw[bk][3]};
                C = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h16x8, w), bq[bk], C, 0, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) S[i] = C[i];
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) S[i] = 0.f;
            const uint32_t k64 = 0x64646464u;
#pragma unroll
            for (int bk = 0; bk < NBK; ++bk) {
                uint32_t a[4];
                if constexpr (FMT == LW_Q8_0) {
                    const uint32_t w0 = t.kw[bk][0] ^ 0x80808080u, w1 = t.kw[bk][1] ^ 0x80808080u;
                    a[0] = __builtin_amdgcn_perm(k64, w0, 0x04010400u);
                    a[1] = __builtin_amdgcn_perm(k64, w0, 0x04030402u);
                    a[2] = __builtin_amdgcn_perm(k64, w1, 0x04010400u);
                    a[3] = __builtin_amdgcn_perm(k64, w1, 0x04030402u);
                } else {
                    const uint32_t lo = opaque(t.kw[bk][0] & 0x0F0F0F0Fu);
                    const uint32_t hi = opaque((t.kw[bk][0] >> 4) & 0x0F0F0F0Fu);
                    a[0] = __builtin_amdgcn_perm(k64, lo, 0x04010400u);
                    a[1] = __builtin_amdgcn_perm(k64, lo, 0x04030402u);
                    a[2] = __builtin_amdgcn_perm(k64, hi, 0x04010400u);
                    a[3] = __builtin_amdgcn_perm(k64, hi, 0x04030402u);
                }
                const f32x4 C0 = {cb[bk], cb[bk], cb[bk], cb[bk]};
                const f32x4 C = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h16x8, a), bq[bk], C0, 0, 0, 0);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t sw = t.ks[i][bk >> 1];
                    const float d = half_bits_to_float((bk & 1) ? sw >> 16 : sw & 0xFFFFu);
                    S[i] = __builtin_fmaf(d, C[i], S[i]);
                }
            }
        }
        // the high part's column n plus the low part's column G + n
        float s[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float tot = S[i] + dpp_move<0x100 + G>(S[i]);  // row_shl: lane n reads lane n + G
            s[i] = b + 4 * gq + i < j1 ? tot * sc : -INFINITY;
        }
        float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
        mx = fmaxf(mx, partner<16>(mx));
        mx = fmaxf(mx, partner<32>(mx));  // the tile's maximum of head n (its first row is valid)
        const float mn = fmaxf(m_l, mx);
        if (__builtin_amdgcn_ballot_w64(n < G && mn != m_l)) {  // a head's maximum grew
            const float alpha = __builtin_amdgcn_exp2f(m_l - mn);  // m = -inf: 0; unchanged: 1
            l_l *= alpha;
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float ah = __builtin_bit_cast(
                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), h));  // lane h: head h
#pragma unroll
                for (int i = 0; i < DPL; ++i) acc[h][i] *= ah;
            }
        }
        m_l = mn;
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(s[i] - m_l);  // masked: 0
        l_l += (p[0] + p[1]) + (p[2] + p[3]);
        if (n < G) {
#pragma unroll
            for (int i = 0; i < 4; ++i) pw[wave][4 * gq + i][n] = p[i];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // outputs: the value layout, BPT batches of RPW positions
#pragma unroll
        for (int j = 0; j < BPT; ++j) {
            float ph[G];
#pragma unroll
            for (int h = 0; h < G; ++h) ph[h] = pw[wave][j * RPW + r][h];
            float vv[DPL], va;
            RW::decode(t.v[j], sh, vv, va);
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float pa = RW::kAffine ? ph[h] * va : ph[h];
#pragma unroll
                for (int i = 0; i < DPL; ++i) acc[h][i] = __builtin_fmaf(pa, vv[i], acc[h][i]);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    // tiles b, b + 64, ... of this wave, two in flight (as the split kernel's
    // sets: unconditional loads, one exit, wave-uniform trip count)
    constexpr int kTileStep = kAttnWaves * 16;
    int b = j0 + wave * 16;
    if (b < j1) {
        const int nt = (j1 - b + kTileStep - 1) / kTileStep;
        Tile ta, tb;
        load_tile(b, ta);
        for (int t = 2; t <= nt; t += 2) {
            load_tile(b + kTileStep, tb);
            use_tile(b, ta);
            load_tile(b + 2 * kTileStep, ta);
            use_tile(b + kTileStep, tb);
            b += 2 * kTileStep;
        }
        if (nt & 1) use_tile(b, ta);
    }

    {
        float v[G * DPL];
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int i = 0; i < DPL; ++i) v[h * DPL + i] = acc[h][i];
        wave_outputs_to_lds<D, G, DPL>(v, red[wave], lane, c);
    }
    // head n's weight sum over the four lane groups; lane h < G (gq = 0) writes head h
    l_l += partner<16>(l_l);
    l_l += partner<32>(l_l);
    if (lane < G) {
        red[wave][lane][D] = m_l;
        red[wave][lane][D + 1] = l_l;
    }
    __syncthreads();
    merge_waves<D, G>(red, ws + ((int64_t)split * n_heads + (int64_t)g * G) * (D + 2));
}

// out[h][d] = sum_s exp(m_s - M) acc_s[d] / sum_s exp(m_s - M) l_s. One
// workgroup per head; thread (d, sg) takes output d of the splits sg,
// sg + SG, ...: their maxima and partials are loaded together (one round
// trip for up to U splits per thread), summed against the thread's own
// running maximum, and the SG groups merged through LDS with one more
// rescale each (the same merge as the split kernel's waves).
constexpr int kCombThreads = 512;

template <int D>
__global__ void __launch_bounds__(kCombThreads) attn_combine_kernel(const float* __restrict__ ws,
                                                                   float* __restrict__ out, int n_heads, int splits) {
    constexpr int SG = kCombThreads / D;  // split groups
    constexpr int U = 16;                 // splits per thread and round
    __shared__ float part[SG][D + 2];     // group sums of output d; [D]: the group's maximum, [D + 1]: its l
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* base = ws + (int64_t)h * (D + 2);
    const int64_t stride = (int64_t)n_heads * (D + 2);
    const int sg = tid / D, d0 = tid - sg * D;
    const bool with_l = d0 == 1;  // thread d = 1 also sums l (slot D + 1)
    float M = -INFINITY, o = 0.f, ol = 0.f;
    for (int s = sg; s < splits; s += U * SG) {
        float mv[U], v[U], vl[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int su = s + u * SG;
            const bool ok = su < splits;
            const float* p = base + (int64_t)(ok ? su : 0) * stride;
            mv[u] = ok ? p[D] : -INFINITY;
            v[u] = ok ? p[d0] : 0.f;
            vl[u] = ok && with_l ? p[D + 1] : 0.f;
        }
        float mc = M;
#pragma unroll
        for (int u = 0; u < U; ++u) mc = fmaxf(mc, mv[u]);
        // every split has a position, so mc is finite from the first round on
        const float a = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - mc);
        o *= a;
        ol *= a;
        M = mc;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float w = mv[u] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mv[u] - M);
            o = __builtin_fmaf(w, v[u], o);
            ol = __builtin_fmaf(w, vl[u], ol);
        }
    }
    part[sg][d0] = o;
    if (d0 == 0) part[sg][D] = M;  // -inf for a group without splits
    if (with_l) part[sg][D + 1] = ol;
    __syncthreads();
    if (tid < D) {
        float Mh = -INFINITY;
#pragma unroll
        for (int g = 0; g < SG; ++g) Mh = fmaxf(Mh, part[g][D]);
        float y = 0.f, L = 0.f;
#pragma unroll
        for (int g = 0; g < SG; ++g) {
            const float mg = part[g][D];
            const float w = mg == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mg - Mh);
            y = __builtin_fmaf(w, part[g][tid], y);
            L = __builtin_fmaf(w, part[g][D + 1], L);
        }
        out[(int64_t)h * D + tid] = y / L;
    }
}

template <int FMT, int D, int G>
hipError_t launch_g(const float* q, const uint8_t* K, const uint8_t* V, float* out, int64_t n_heads, int64_t n_kv,
                    int64_t kv_len, float scale, const AttnPlan& pl, float* ws, hipStream_t stream) {
    const Planes p = planes_of(FMT, n_kv * kv_len * D);
    // f16, Q8_0 and Q4_0 caches with more than one 64-position round per
    // workgroup: scores on the matrix cores (with a single round its query
    // preparation is not repaid)
    constexpr bool kMf = FMT == LW_F16 || FMT == LW_Q8_0 || FMT == LW_Q4_0;
    if (kMf && pl.rps > kMfMinRps) {
        constexpr int FM = kMf ? FMT : LW_F16;  // instantiated for the three formats only
        if (query_only(kernel_name<Name_attn_mf_kernel, FM, D, G>(), 2)) return hipSuccess;
        hipLaunchKernelGGL((attn_mf_kernel<FM, D, G>), dim3((unsigned)n_kv, (unsigned)pl.splits),
                           dim3(kAttnThreads), 0, stream, q, K, V, p.off1, (int)kv_len, (int)n_heads, scale,
                           (int)pl.rps, ws);
    } else {
        if (query_only(kernel_name<Name_attn_split_kernel, FMT, D, G>(), 2)) return hipSuccess;
        hipLaunchKernelGGL((attn_split_kernel<FMT, D, G>), dim3((unsigned)n_kv, (unsigned)pl.splits),
                           dim3(kAttnThreads), 0, stream, q, K, V, p.off1, p.off2, p.off3, (int)kv_len, (int)n_heads,
                           scale, (int)pl.rps, ws);
    }
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
    // about one workgroup per compute unit, at least 64 positions each (the
    // per-wave reductions are paid once per split). Measured against two
    // per unit (32 query heads over 8 KV heads of 128, q8_0): 8192 positions
    // 14.2 -> 12.9 us, 32768: 25.7 -> 23.2 (longer loops per wave, half the
    // partial results to combine); three or four per unit are slower.
    const int64_t by_len = (kv_len + 63) / 64;
    const int64_t by_chip = (256 + n_kv - 1) / n_kv;
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
