// Few-token product on the matrix cores for the 4-bit formats (2 <= n_tok <= 16).
//
// Y[t][r] = sum_k value(W, r*K + k) * X[t][k]: the decode product of Sec. 2.1
// for a small batch of tokens, with the weights streamed from HBM exactly once
// and dequantized in registers (Sec. 3.3). The contraction runs on
// v_mfma_f32_16x16x32_bf16 (D[16x16] += A[16x32] . B[32x16]) with one MFMA K
// step per 32-element block, so each block's scale applies to its own partial
// product: A = X (the token rows), B = the codes of 16 weight rows.
// Two kernels: multitok_pk_kernel (up to 8 tokens: high and low parts of the
// tokens packed into the 16 A rows, codes read as whole 128-byte lines and
// regrouped through LDS) and multitok_kernel (9..16 tokens: A rows are
// tokens, high and low parts in two MFMAs).
//
// Precision (the reading shared by the matrix-core paths): B holds the exact
// bf16 of the biased code 128 + q (bit pattern 0x4300 | q); X is split into a
// bf16 high part and a bf16 low part, both multiplied; per block
// y += c1 * (P + k * S) - dm * S, with S the block sum of the operand actually
// multiplied (hi + lo). k * S comes from the same A operands against a B of
// the constant k (exact in bf16) and is the accumulator P starts from:
//   Q4_0:     w = d (q - 8)         -> c1 = d,    k = -136, dm = 0
//   Q4_K:     w = d sc q - dmin m   -> c1 = d sc, k = -128, dm = dmin m
//   Q4_1:     w = d q + m           -> c1 = d,    k = -128, dm = -m
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

int cu_count_mt() {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
        return 256;
    return v;
}

// 4 x 4 transpose across the four 16-lane groups: lane (g, i) holds words
// w0..w3 of block g of its row; afterwards word j of the result is word g of
// block j (v_permlane32_swap, v_permlane16_swap).
__device__ __forceinline__ u32x4 quad_transpose(u32x4 w) {
    const auto s02 = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
    const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    return u32x4{s01[0], s01[1], s23[0], s23[1]};
}

// Scale data of a step (4 blocks of one weight row, inside one super-block).
template <int FMT>
struct StepScale;

template <>
struct StepScale<LW_Q4_0> {
    uint32_t a, b;  // binary16 d of the 4 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t row, uint32_t K, uint32_t s, int) {
        const uint2 v = *reinterpret_cast<const uint2*>(P1 + 2 * (row * (K / 32u) + 4u * s));
        a = v.x;
        b = v.y;
    }
    // c1 of the step's blocks (d), and dm = 0
    __device__ void coef(uint32_t, int, float* c1, float* dm) const {
        c1[0] = half_bits_to_float(a & 0xFFFFu);
        c1[1] = half_bits_to_float(a >> 16);
        c1[2] = half_bits_to_float(b & 0xFFFFu);
        c1[3] = half_bits_to_float(b >> 16);
        dm[0] = dm[1] = dm[2] = dm[3] = 0.f;
    }
};

template <>
struct StepScale<LW_Q4_1> {
    u32x4 v;  // {binary16 d, binary16 m} of the 4 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t row, uint32_t K, uint32_t s, int) {
        v = *reinterpret_cast<const u32x4*>(P1 + 4 * (row * (K / 32u) + 4u * s));
    }
    // c1 = d and dm = -m / 128 of the step's blocks
    __device__ void coef(uint32_t, int, float* c1, float* dm) const {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            c1[i] = half_bits_to_float(v[i] & 0xFFFFu);
            dm[i] = half_bits_to_float(v[i] >> 16) * (-1.0f / 128.0f);
        }
    }
};

template <>
struct StepScale<LW_Q4_K> {
    uint32_t r0, r1, r2, dd;  // the super-block's 96-bit record and {d, dmin}
    __device__ void load(const uint8_t* P1, const uint8_t* P2, uint64_t row, uint32_t K, uint32_t s, int) {
        const uint64_t sb = row * (K / 256u) + (s >> 1);
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(P1 + 12 * sb);
        r0 = rec[0];
        r1 = rec[1];
        r2 = rec[2];
        dd = *reinterpret_cast<const uint32_t*>(P2 + 4 * sb);
    }
    // c1 = d*sc_j and dm = dmin*m_j/128 of the step's blocks, sub-blocks
    // j = 4(s&1) + 0..3 of the super-block: sc_j at record bit 6j, m_j at
    // bit 48 + 6j, cut out of one rotated word or one word pair each.
    __device__ void coef(uint32_t s, int, float* c1, float* dm) const {
        const float d = half_bits_to_float(dd & 0xFFFFu), dmin = half_bits_to_float(dd >> 16) * (1.0f / 128.0f);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t j = 4u * (s & 1u) + (uint32_t)i;
            const uint32_t ts = 6u * j, tm = 16u + 6u * j;
            const uint32_t sc_w = __builtin_amdgcn_alignbit(r1, ts < 32u ? r0 : r1, ts & 31u);
            const uint32_t m_w = __builtin_amdgcn_alignbit(r2, tm < 32u ? r1 : r2, tm & 31u);
            c1[i] = d * (float)(sc_w & 63u);
            dm[i] = dmin * (float)(m_w & 63u);
        }
    }
};

template <int FMT, int NX, int RG>
struct Stage {
    u32x4 codes[RG];
    StepScale<FMT> sc[RG];
    float4 xv[NX];
};

// Few-token product with whole-block MFMAs: D = X . W^T per 32-element block,
// A = X (token rows), B = the codes of 16 weight rows. A step is 4 blocks
// (128 columns) of RG row tiles. Lane (g, i) loads block 4s+g of row i of
// each tile (one 16-byte load, a whole block), and a transpose across the
// lane groups gives it word g of each of the 4 blocks, its B slice (elements
// 4g..4g+3 and 16+4g..16+4g+3) for the 4 MFMAs. D lands as D[4g+v][i]: one
// weight row per lane, so each lane applies its row's block scale with no
// exchange.
// A rows are tokens (up to 16; rows of tokens >= n_tok are zero): the bf16
// high parts in one operand, the low parts in a second, two MFMAs per block.
// The bias correction k * S enters as the MFMA accumulator: C = A . B_k, with
// B_k the constant bf16 k, per block, shared by the row tiles. Then
// y += c1 * P per block (Q4_K: also + dmin m / 128 * C, C being -128 S).
// X: every step, the wave converts its 4 blocks of the n_tok token rows
// densely (lane -> token, block, float4; NX float4 per lane; the loads of one
// block are 128 contiguous bytes), hi/lo bf16 halves into its private LDS
// slice in the A layout, then reads its A operands back. Waves split K; their
// partials are summed through LDS at the end.
template <int FMT, int NX, int RG>
__global__ void __launch_bounds__(64 * kMaxWaves)
    multitok_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                     int64_t K, int ntok, int64_t off1, int64_t off2) {
    extern __shared__ float4 smem4[];
    constexpr int NH = 2;                       // A planes: hi and lo
    constexpr int kSlice = NH * 4 * 64 + 1;     // the wave's LDS slice, in 16-byte slots
    const int nw = blockDim.x >> 6;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n16 = lane & 15, g = lane >> 4;
    const uint32_t K32 = (uint32_t)K;
    const uint8_t* P1 = W + off1;
    const uint8_t* P2 = W + off2;

    const int nsteps = (int)(K / 128);
    const int spw = (nsteps + nw - 1) / nw;
    const int s0 = wave * spw;
    const int s1 = (s0 + spw) < nsteps ? (s0 + spw) : nsteps;

    const int64_t row0 = (int64_t)blockIdx.x * 16 * RG;
    uint64_t row[RG];
    const uint8_t* cp[RG];
#pragma unroll
    for (int q = 0; q < RG; ++q) {
        const int64_t r = row0 + 16 * q + n16;
        row[q] = (uint64_t)(r < M ? r : M - 1);
        cp[q] = W + row[q] * (K32 / 2u) + 16u * g;
    }
    // dense X items: item e of the lane is float4 m of block j of token t
    int xm[NX], xj[NX], xt[NX];
    bool xlive[NX];
    const float* xp[NX];
#pragma unroll
    for (int e = 0; e < NX; ++e) {
        const int idx = lane + 64 * e;
        xm[e] = idx & 7;
        xj[e] = (idx >> 3) & 3;
        xt[e] = idx >> 5;
        xlive[e] = xt[e] < ntok;
        xp[e] = x + (int64_t)(xlive[e] ? xt[e] : ntok - 1) * K + 32 * xj[e] + 4 * xm[e];
    }
    // the wave's A slice: [plane][block j][64 slots] of 16 bytes, then a
    // spare 16 bytes that absorb the writes of padding items. A row n of lane
    // group gg in block j sits in slot 16gg + (n ^ (2gg + (j & 1) + 8(j >> 1))):
    // a permutation of each 16-slot group, so the reads stay conflict-free,
    // which spreads the 8-byte writes of one instruction (items of one token,
    // 4 blocks x 8 float4) over distinct banks.
    auto xslot = [](int gg, int n, int j) { return 16 * gg + (n ^ (2 * gg + (j & 1) + 8 * (j >> 1))); };
    constexpr int kSpare = 2 * (kSlice - 1);
    uint2* xs = reinterpret_cast<uint2*>(smem4 + (size_t)wave * kSlice);
#pragma unroll
    for (int h = 0; h < NH * 4; ++h) {
        xs[2 * (h * 64 + lane)] = uint2{0u, 0u};
        xs[2 * (h * 64 + lane) + 1] = uint2{0u, 0u};
    }

    auto load = [&](Stage<FMT, NX, RG>& st, int s) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < RG; ++q) {
            st.codes[q] = load_codes(cp[q] + 64u * (uint32_t)s);
            st.sc[q].load(P1, P2, row[q], K32, (uint32_t)s, g);
        }
#pragma unroll
        for (int e = 0; e < NX; ++e) st.xv[e] = *reinterpret_cast<const float4*>(xp[e] + 128 * s);
    };

    // bf16 k: -136 (Q4_0: code bias 128 plus the format's offset 8) or -128
    const uint32_t kb = FMT == LW_Q4_0 ? 0xC308C308u : 0xC300C300u;
    const bf16x8 bias_b = __builtin_bit_cast(bf16x8, u32x4{kb, kb, kb, kb});
    f32x4 acc[RG];
#pragma unroll
    for (int q = 0; q < RG; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto consume = [&](const Stage<FMT, NX, RG>& st, int s) __attribute__((always_inline)) {
        // X of the step -> hi/lo halves in the A layout: item (t, j, m) is
        // half m >> 2 of the 16 bytes of lane group m & 3 in block j, A row t
        // of plane 0 (high part) and of plane 1 (low part)
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int e = 0; e < NX; ++e) {
            const float v[4] = {st.xv[e].x, st.xv[e].y, st.xv[e].z, st.xv[e].w};
            typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
            typedef float f32x2 __attribute__((ext_vector_type(2)));
            uint32_t hw[2], lw[2];
#pragma unroll
            for (int p2 = 0; p2 < 2; ++p2) {
                const uint32_t hb = __builtin_bit_cast(
                    uint32_t, __builtin_convertvector((f32x2{v[2 * p2], v[2 * p2 + 1]}), bf16x2));
                const float h0 = __builtin_bit_cast(float, hb << 16), h1 = __builtin_bit_cast(float, hb & 0xFFFF0000u);
                hw[p2] = hb;
                lw[p2] = __builtin_bit_cast(
                    uint32_t, __builtin_convertvector((f32x2{v[2 * p2] - h0, v[2 * p2 + 1] - h1}), bf16x2));
            }
            // an item of a token >= n_tok goes to the slice's spare slot
            const int gg = xm[e] & 3, half = xm[e] >> 2, j = xj[e], t = xt[e];
            const int sh = j * 64 + xslot(gg, t, j);
            const int sl = (4 + j) * 64 + xslot(gg, t, j);
            const int ih = xlive[e] ? 2 * sh + half : kSpare;
            const int il = xlive[e] ? 2 * sl + half : kSpare;
            xs[ih] = uint2{hw[0], hw[1]};
            xs[il] = uint2{lw[0], lw[1]};
        }
        __builtin_amdgcn_wave_barrier();
        bf16x8 a[NH][4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int h = 0; h < NH; ++h)
                a[h][j] = __builtin_bit_cast(bf16x8,
                                             reinterpret_cast<const float4*>(xs)[(h * 4 + j) * 64 + xslot(g, n16, j)]);
        // C = k * (block sums of the multiplied values), in the D layout
        f32x4 C[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            C[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0][j], bias_b, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            C[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1][j], bias_b, C[j], 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < RG; ++q) {
            const u32x4 wq = quad_transpose(st.codes[q]);
            float c1[4], dm[4];
            st.sc[q].coef((uint32_t)s, g, c1, dm);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bf16x8 bq = biased_codes(wq[j]);
                f32x4 P = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0][j], bq, C[j], 0, 0, 0);
                P = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1][j], bq, P, 0, 0, 0);
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float o = __builtin_fmaf(c1[j], P[v], acc[q][v]);
                    if constexpr (FMT != LW_Q4_0) o = __builtin_fmaf(dm[j], C[j][v], o);
                    acc[q][v] = o;
                }
            }
        }
    };

    // Two stages in flight. Every load is issued unconditionally (a step
    // index past the wave's range is clamped to its last step, an in-range
    // reload never consumed), so the compiler's vmcnt waits stay exact and a
    // consume never waits for the refill issued after it.
    const int slast = s1 > s0 ? s1 - 1 : (s0 < nsteps ? s0 : nsteps - 1);
    auto clampst = [&](int st) { return st < s1 ? st : slast; };
    Stage<FMT, NX, RG> sa, sb;
    load(sa, clampst(s0));
    load(sb, clampst(s0 + 1));
    int s = s0;
    for (; s + 4 <= s1; s += 2) {
        consume(sa, s);
        __builtin_amdgcn_sched_barrier(0);
        load(sa, s + 2);
        __builtin_amdgcn_sched_barrier(0);
        consume(sb, s + 1);
        __builtin_amdgcn_sched_barrier(0);
        load(sb, s + 3);
        __builtin_amdgcn_sched_barrier(0);
    }
    // the last 0..3 steps
    if (s < s1) consume(sa, s);
    load(sa, clampst(s + 2));
    if (s + 1 < s1) consume(sb, s + 1);
    if (s + 2 < s1) consume(sa, s + 2);

    // sum the partials of the waves: lane holds D rows (tokens) 4g + v of
    // weight row 16q + n16
    __syncthreads();
    constexpr int kRows = 16 * RG;
    float* red = reinterpret_cast<float*>(smem4);  // [nw][16 D rows][kRows]
#pragma unroll
    for (int q = 0; q < RG; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[(wave * 16 + 4 * g + v) * kRows + 16 * q + n16] = acc[q][v];
    __syncthreads();
    for (int it = tid; it < 16 * kRows; it += blockDim.x) {
        const int t = it / kRows, r = it % kRows;
        if (t < ntok && row0 + r < M) {
            float o = 0.f;
            for (int p = 0; p < nw; ++p) o += red[(p * 16 + t) * kRows + r];
            y[(int64_t)t * M + row0 + r] = o;
        }
    }
}

// Scale data of a pair-step (8 blocks, 256 columns, of one weight row; for
// Q4_K exactly one super-block).
template <int FMT>
struct PairScale;

template <>
struct PairScale<LW_Q4_0> {
    u32x4 w;  // binary16 d of the 8 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t row, uint32_t K, uint32_t ps) {
        w = *reinterpret_cast<const u32x4*>(P1 + 2 * (row * (K / 32u) + 8u * ps));
    }
    // c1 of blocks 4h..4h+3 (d)
    __device__ void coef(int h, float* c1, float*) const {
        const uint32_t a = h ? w[2] : w[0], b = h ? w[3] : w[1];
        c1[0] = half_bits_to_float(a & 0xFFFFu);
        c1[1] = half_bits_to_float(a >> 16);
        c1[2] = half_bits_to_float(b & 0xFFFFu);
        c1[3] = half_bits_to_float(b >> 16);
    }
};

template <>
struct PairScale<LW_Q4_1> {
    u32x4 v[2];  // {binary16 d, binary16 m} of the 8 blocks
    __device__ void load(const uint8_t* P1, const uint8_t*, uint64_t row, uint32_t K, uint32_t ps) {
        const uint8_t* p = P1 + 4 * (row * (K / 32u) + 8u * ps);
        v[0] = *reinterpret_cast<const u32x4*>(p);
        v[1] = *reinterpret_cast<const u32x4*>(p + 16);
    }
    // c1 = d and dm = -m / 128 of blocks 4h..4h+3
    __device__ void coef(int h, float* c1, float* dm) const {
        const u32x4 w = h ? v[1] : v[0];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            c1[i] = half_bits_to_float(w[i] & 0xFFFFu);
            dm[i] = half_bits_to_float(w[i] >> 16) * (-1.0f / 128.0f);
        }
    }
};

template <>
struct PairScale<LW_Q4_K> {
    uint32_t r0, r1, r2, dd;  // the super-block's 96-bit record and {d, dmin}
    __device__ void load(const uint8_t* P1, const uint8_t* P2, uint64_t row, uint32_t K, uint32_t ps) {
        const uint64_t sb = row * (K / 256u) + ps;
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(P1 + 12 * sb);
        r0 = rec[0];
        r1 = rec[1];
        r2 = rec[2];
        dd = *reinterpret_cast<const uint32_t*>(P2 + 4 * sb);
    }
    // c1 = d*sc_j and dm = dmin*m_j/128 of sub-blocks j = 4h..4h+3: sc_j at
    // record bit 6j, m_j at bit 48 + 6j (fixed positions once h is known)
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

template <int FMT, int NX, int RG>
struct PairStage {
    u32x4 codes[RG][2];
    PairScale<FMT> sc[RG];
    float4 xv[2][NX];
};

// Few-token product for n_tok <= 8 with whole-line code loads. Same MFMA
// scheme as multitok_kernel with packed A rows (hi parts of tokens 0..7 in
// rows 0..7, lo parts in rows 8..15), but the unit of work is a pair-step of
// 8 blocks (256 columns), and the codes of a 16-row tile come in as two
// loads of 8 rows x 128 bytes (lane 8k + m: row 8r + k, block m ^ k ^ r), so
// every load instruction reads whole 128-byte lines. The wave stages them in
// its private LDS (slot 64r + lane) and reads them back as lane (g, i) <-
// block 4h + g of row i (slot 64r + 8k + (b ^ k ^ r) for row i = 8r + k: a
// permutation within each 8-slot row that keeps the 16-lane groups of a read
// on distinct banks). Scales come once per pair-step.
template <int FMT, int NX, int RG>
__global__ void __launch_bounds__(64 * kMaxWaves)
    multitok_pk_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y, int64_t M,
                        int64_t K, int ntok, int64_t off1, int64_t off2) {
    extern __shared__ float4 smem4[];
    constexpr int kXSlots = 4 * 64 + 1;             // A slice of one half (4 blocks x 64 slots) + spare
    constexpr int kSlice = kXSlots + RG * 128;       // + codes staging, 2 KiB per tile
    const int nw = blockDim.x >> 6;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n16 = lane & 15, g = lane >> 4;
    const uint32_t K32 = (uint32_t)K;
    const uint8_t* P1 = W + off1;
    const uint8_t* P2 = W + off2;

    const int nps = (int)(K / 256);
    const int ppw = (nps + nw - 1) / nw;
    const int p0 = wave * ppw;
    const int p1 = (p0 + ppw) < nps ? (p0 + ppw) : nps;

    const int64_t row0 = (int64_t)blockIdx.x * 16 * RG;
    uint64_t row[RG];
    const uint8_t* cp[RG][2];
    const int ck = lane >> 3, cm = lane & 7;
#pragma unroll
    for (int q = 0; q < RG; ++q) {
        const int64_t r = row0 + 16 * q + n16;
        row[q] = (uint64_t)(r < M ? r : M - 1);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int64_t rr = row0 + 16 * q + 8 * h + ck;
            const uint64_t rc = (uint64_t)(rr < M ? rr : M - 1);
            cp[q][h] = W + rc * (K32 / 2u) + 16u * (uint32_t)(cm ^ ck ^ h);
        }
    }
    int xm[NX], xj[NX], xt[NX];
    bool xlive[NX];
    const float* xp[NX];
#pragma unroll
    for (int e = 0; e < NX; ++e) {
        const int idx = lane + 64 * e;
        xm[e] = idx & 7;
        xj[e] = (idx >> 3) & 3;
        xt[e] = idx >> 5;
        xlive[e] = xt[e] < ntok;
        xp[e] = x + (int64_t)(xlive[e] ? xt[e] : ntok - 1) * K + 32 * xj[e] + 4 * xm[e];
    }
    auto xslot = [](int gg, int n, int j) { return 16 * gg + (n ^ (2 * gg + (j & 1) + 8 * (j >> 1))); };
    constexpr int kSpare = 2 * (kXSlots - 1);
    float4* wbase = smem4 + (size_t)wave * kSlice;
    uint2* xs = reinterpret_cast<uint2*>(wbase);
    float4* cs = wbase + kXSlots;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        xs[2 * (h * 64 + lane)] = uint2{0u, 0u};
        xs[2 * (h * 64 + lane) + 1] = uint2{0u, 0u};
    }
    // read slot of lane (g, n16) for half h of a staged tile
    const int rd0 = 64 * (n16 >> 3) + 8 * (n16 & 7);
    const int rdx = (n16 & 7) ^ (n16 >> 3);

    auto load = [&](PairStage<FMT, NX, RG>& st, int ps) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < RG; ++q) {
            st.codes[q][0] = load_codes(cp[q][0] + 128u * (uint32_t)ps);
            st.codes[q][1] = load_codes(cp[q][1] + 128u * (uint32_t)ps);
            st.sc[q].load(P1, P2, row[q], K32, (uint32_t)ps);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < NX; ++e)
                st.xv[h][e] = *reinterpret_cast<const float4*>(xp[e] + 256 * ps + 128 * h);
    };

    const uint32_t kb = FMT == LW_Q4_0 ? 0xC308C308u : 0xC300C300u;
    const bf16x8 bias_b = __builtin_bit_cast(bf16x8, u32x4{kb, kb, kb, kb});
    f32x4 acc[RG];
#pragma unroll
    for (int q = 0; q < RG; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto consume = [&](const PairStage<FMT, NX, RG>& st) __attribute__((always_inline)) {
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < RG; ++q) {
            cs[128 * q + lane] = __builtin_bit_cast(float4, st.codes[q][0]);
            cs[128 * q + 64 + lane] = __builtin_bit_cast(float4, st.codes[q][1]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            // one half at a time: the scheduler may not overlap the halves
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int e = 0; e < NX; ++e) {
                const float v[4] = {st.xv[h][e].x, st.xv[h][e].y, st.xv[h][e].z, st.xv[h][e].w};
                typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
                typedef float f32x2 __attribute__((ext_vector_type(2)));
                uint32_t hw[2], lw[2];
#pragma unroll
                for (int p2 = 0; p2 < 2; ++p2) {
                    const uint32_t hb = __builtin_bit_cast(
                        uint32_t, __builtin_convertvector((f32x2{v[2 * p2], v[2 * p2 + 1]}), bf16x2));
                    const float h0 = __builtin_bit_cast(float, hb << 16),
                                h1 = __builtin_bit_cast(float, hb & 0xFFFF0000u);
                    hw[p2] = hb;
                    lw[p2] = __builtin_bit_cast(
                        uint32_t, __builtin_convertvector((f32x2{v[2 * p2] - h0, v[2 * p2 + 1] - h1}), bf16x2));
                }
                const int gg = xm[e] & 3, half = xm[e] >> 2, j = xj[e], t = xt[e];
                const int ih = xlive[e] ? 2 * (j * 64 + xslot(gg, t, j)) + half : kSpare;
                const int il = xlive[e] ? 2 * (j * 64 + xslot(gg, 8 + t, j)) + half : kSpare;
                xs[ih] = uint2{hw[0], hw[1]};
                xs[il] = uint2{lw[0], lw[1]};
            }
            __builtin_amdgcn_wave_barrier();
            bf16x8 a[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                a[j] = __builtin_bit_cast(bf16x8, reinterpret_cast<const float4*>(xs)[j * 64 + xslot(g, n16, j)]);
            f32x4 C[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                C[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], bias_b, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
#pragma unroll
            for (int q = 0; q < RG; ++q) {
                const u32x4 blk = __builtin_bit_cast(u32x4, cs[128 * q + rd0 + ((4 * h + g) ^ rdx)]);
                const u32x4 wq = quad_transpose(blk);
                f32x4 P[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    P[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], biased_codes(wq[j]), C[j], 0, 0, 0);
                float c1[4], dm[4];
                st.sc[q].coef(h, c1, dm);
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float o = __builtin_fmaf(c1[j], P[j][v], acc[q][v]);
                        if constexpr (FMT != LW_Q4_0) o = __builtin_fmaf(dm[j], C[j][v], o);
                        acc[q][v] = o;
                    }
            }
        }
    };

    // Two pair-steps in flight, loads issued unconditionally (see
    // multitok_kernel); the tail issues only loads that are consumed.
    auto clampps = [&](int v) { return v < p1 ? v : (p1 > p0 ? p1 - 1 : (p0 < nps ? p0 : nps - 1)); };
    PairStage<FMT, NX, RG> sa, sb;
    load(sa, clampps(p0));
    load(sb, clampps(p0 + 1));
    int ps = p0;
    for (; ps + 4 <= p1; ps += 2) {
        consume(sa);
        __builtin_amdgcn_sched_barrier(0);
        load(sa, ps + 2);
        __builtin_amdgcn_sched_barrier(0);
        consume(sb);
        __builtin_amdgcn_sched_barrier(0);
        load(sb, ps + 3);
        __builtin_amdgcn_sched_barrier(0);
    }
    // the last 0..3 pair-steps (sa holds ps, sb holds ps + 1)
    const int rem = p1 - ps;
    if (rem == 3) {
        consume(sa);
        __builtin_amdgcn_sched_barrier(0);
        load(sa, ps + 2);
        __builtin_amdgcn_sched_barrier(0);
        consume(sb);
        consume(sa);
    } else {
        if (rem >= 1) consume(sa);
        if (rem >= 2) consume(sb);
    }

    // sum the partials of the waves and the high and low D rows of a token
    __syncthreads();
    constexpr int kRows = 16 * RG;
    float* red = reinterpret_cast<float*>(smem4);  // [nw][16 D rows][kRows]
#pragma unroll
    for (int q = 0; q < RG; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[(wave * 16 + 4 * g + v) * kRows + 16 * q + n16] = acc[q][v];
    __syncthreads();
    for (int it = tid; it < 8 * kRows; it += blockDim.x) {
        const int t = it / kRows, r = it % kRows;
        if (t < ntok && row0 + r < M) {
            float o = 0.f;
            for (int p = 0; p < nw; ++p) o += red[(p * 16 + t) * kRows + r] + red[(p * 16 + 8 + t) * kRows + r];
            y[(int64_t)t * M + row0 + r] = o;
        }
    }
}

struct Name_multitok_pk_kernel {
    static constexpr const char* base = "multitok_pk_kernel";
};

template <int FMT, int NX, int RG>
hipError_t launch_pk(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                      const Planes& p, int nw, hipStream_t stream) {
    const int64_t grid = (M + 16 * RG - 1) / (16 * RG);
    if (grid > 0x7fffffff || nw < 1 || nw > kMaxWaves) return hipErrorInvalidConfiguration;
    if (n_tok > 8 || 32 * n_tok > 64 * NX || K % 256) return hipErrorInvalidValue;
    size_t lds = (size_t)nw * (4 * 64 + 1 + RG * 128) * 16;  // A slice + codes staging per wave
    const size_t red = (size_t)nw * 16 * (16 * RG) * 4;
    if (lds < red) lds = red;
    if (query_only(kernel_name<Name_multitok_pk_kernel, FMT, NX, RG>())) return hipSuccess;
    hipLaunchKernelGGL((multitok_pk_kernel<FMT, NX, RG>), dim3((unsigned)grid), dim3(64 * nw), lds, stream, W, x, y,
                       M, K, (int)n_tok, p.off1, p.off2);
    return hipGetLastError();
}

template <int FMT, int NX, int RG>
hipError_t launch_mt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                      const Planes& p, int nw, hipStream_t stream) {
    const int64_t grid = (M + 16 * RG - 1) / (16 * RG);
    if (grid > 0x7fffffff || nw < 1 || nw > kMaxWaves) return hipErrorInvalidConfiguration;
    if (n_tok > 16 || 32 * n_tok > 64 * NX) return hipErrorInvalidValue;
    size_t lds = (size_t)nw * 513 * 16;                       // A slices, 8 KiB + 16 B per wave
    const size_t red = (size_t)nw * 16 * (16 * RG) * 4;       // final partial sums
    if (lds < red) lds = red;
    if (query_only(kernel_name<Name_multitok_kernel, FMT, NX, RG>())) return hipSuccess;
    hipLaunchKernelGGL((multitok_kernel<FMT, NX, RG>), dim3((unsigned)grid), dim3(64 * nw), lds, stream, W, x, y,
                       M, K, (int)n_tok, p.off1, p.off2);
    return hipGetLastError();
}

template <int FMT, int RG>
hipError_t launch_rg(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                      const Planes& p, int nw, hipStream_t stream) {
    // up to 8 tokens: the pair-step kernel (not for Q4_K with two tiles per
    // wave, whose live state overflows the register file); 32 n_tok floats
    // per step over 64 lanes, in float4s
    if constexpr (FMT == LW_Q4_0 || RG == 1) {
        if (n_tok <= 4) return launch_pk<FMT, 2, RG>(W, x, y, M, K, n_tok, p, nw, stream);
        if (n_tok <= 8) return launch_pk<FMT, 4, RG>(W, x, y, M, K, n_tok, p, nw, stream);
    }
    return launch_mt<FMT, 8, RG>(W, x, y, M, K, n_tok, p, nw, stream);
}

template <int FMT>
hipError_t launch_f(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                     const Planes& p, hipStream_t stream) {
    const int64_t cus = cu_count_mt();
    const bool rg2 = (M + 31) / 32 >= cus;
    const int64_t wgs = rg2 ? (M + 31) / 32 : (M + 15) / 16;
    const int nw = wgs >= 2 * cus ? 4 : 8;
    if (n_tok <= 8 && FMT != LW_Q4_0) return launch_rg<FMT, 1>(W, x, y, M, K, n_tok, p, nw, stream);
    return rg2 ? launch_rg<FMT, 2>(W, x, y, M, K, n_tok, p, nw, stream)
               : launch_rg<FMT, 1>(W, x, y, M, K, n_tok, p, nw, stream);
}

}  // namespace

bool multitok_supported(int fmt, int64_t n_tok) {
    return (fmt == LW_Q4_0 || fmt == LW_Q4_K || fmt == LW_Q4_1) && n_tok >= 2 && n_tok <= 16;
}

hipError_t launch_multitok(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                           int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_Q4_0: return launch_f<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_f<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_1: return launch_f<LW_Q4_1>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
