// Prefill product of LW_MXFP4 weights on MI355X's native fp4 matrix cores.
//
// y[t][r] = sum_k value(W, r*K + k) * x[t][k] with value = e2m1(q) * 2^(E-127),
// the mxfp4 format of Sec. 2.2 and Appendix B (4-bit e2m1 floats sharing one
// power-of-two exponent per 32). The paper emulates this format in software;
// gfx950's v_mfma_scale_f32_32x32x64_f8f6f4 multiplies e2m1 codes directly and
// applies one e8m0 scale per 32 codes inside the instruction, so the weights
// go to the matrix cores exactly as stored (16 code bytes and one exponent
// byte per block): the dequantize-on-load step of Sec. 3.3 becomes part of the
// instruction, and no per-block scaling follows it.
//
// Activations. The instruction's other operand is a 4-, 6- or 8-bit float with
// its own e8m0 scale per 32. x (float32) is split into kPieces e2m3 (fp6)
// pieces. Per 32-element block, with r_0 = x,
//   S_p     = floor(log2 max|r_p|) - 1, clamped to -127 (max|r_p| * 2^-S_p in [2, 4)),
//   c_p     = r_p * 2^-S_p rounded to the nearest e2m3 value (ties to even),
//   r_{p+1} = r_p - c_p * 2^S_p   (exact in float32),
// and every piece keeps four more bits: the e2m3 grid below 4 has steps of
// 1/8 (below 2) and 1/4, so max|r_{p+1}| <= 2^-4 max|r_p| per block, and
// |x - sum_p c_p 2^S_p| <= 2^-16 * (the block's largest |x|). The product is
// sum_p W . (c_p 2^S_p): kPieces instructions per operand pair, accumulated in
// float32 by the matrix core. The fp4 x fp6 form issues at the fp4 rate
// (about 7.8 PFLOP/s measured, twice the fp4 x fp8 form's). The matrix core
// sums the 64 products of one instruction in its own (not IEEE float32)
// order and precision; its error per instruction measured below 2^-12.5 of
// the products' absolute sum. Activations must be finite and below 2^126 in
// magnitude (a larger block's scale would leave the e8m0 range).
//
// Operand layout of the 32 x 32 x 64 form (measured on the GPU): lane l
// supplies row (fp4 operand) or column (fp6 operand) l % 32 at the 32
// consecutive K indices 32 (l / 32) + j, j = 0..31, packed from bit 0 up
// (nibble j of 16 bytes; 6-bit field j of 24 bytes), and its scale byte
// scales exactly those 32. The result D[i][j] lands in lane j + 32 ((i / 4) % 2),
// register 4 (i / 8) + i % 4. Nibble j of a stored block is element
// j / 2 + 16 (j % 2) (the Q4 byte order), so the pieces are packed in that
// same element order and no weight code is moved or decoded.
//
// Launches: xsplit_kernel writes the pieces of every (token, block) to the
// caller's workspace once per call; fp4mm_kernel runs the tiled product;
// where K is split, each split writes its partial results to the workspace
// and ksum_kernel adds them into y. Workgroup tile: 32 RT NW weight rows x 64
// tokens (8 waves, two per SIMD); each wave 32 RT rows (RT 32-row tiles) x 64
// tokens (two 32-token tiles). K advances in stages of four blocks (two K
// windows of 64: lane half h takes blocks 2h + j of the stage in window j);
// the stage's pieces of the 64 tokens are staged in LDS (double buffered),
// the weight codes go from global memory straight to registers. Tile order
// and the XCD grouping are those of the other prefill kernels.
#include <type_traits>

#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

struct Name_fp4mm_kernel {
    static constexpr const char* base = "fp4mm_kernel";
};

constexpr int kPieces = 4;  // e2m3 pieces of the activations
constexpr int kPB = 24;     // bytes of one block's 32 six-bit codes
constexpr int kBN = 64;     // tokens per workgroup
#ifndef LW_FP4_SB
#define LW_FP4_SB 4
#endif
constexpr int kSB = LW_FP4_SB;  // blocks per stage
constexpr int kWS = kSB / 2;    // K windows of 64 per stage
#ifndef LW_FP4_NW
#define LW_FP4_NW 8
#define LW_FP4_RT 2
#endif
constexpr int kNW = LW_FP4_NW;           // waves per workgroup
constexpr int kRT = LW_FP4_RT;           // 32-row tiles per wave
constexpr int kBM = 32 * kRT * kNW;      // weight rows per workgroup

// Tile and K-split plan of a call (row tiles of BM rows, token tiles of kBN)
// and its workspace, token-tile major so that one stage of one workgroup is
// one contiguous run: codes [ntp / kBN][K/32][kPieces][kBN][24 bytes], the
// scale bytes [ntp / kBN][K/32][kPieces][kBN] at s_off, and with K splits
// their float32 partial results [ks][n_tok][M] at p_off (summed into y by a
// last launch). ntp = n_tok rounded up to kBN (the padding tokens are split
// from zeros). The split count is planned for 256 compute units whatever the
// device, so that lw_matvec_workspace_bytes needs no device.
struct XLayout {
    int64_t ntp, nb, s_off, p_off, total;
    GemmSplit sp;
};

XLayout xlayout(int64_t M, int64_t K, int64_t n_tok) {
    XLayout L;
    L.ntp = (n_tok + kBN - 1) / kBN * kBN;
    L.nb = K / 32;
    L.sp = plan_split((M + kBM - 1) / kBM, L.ntp / kBN, K, 256);
    L.s_off = round_up_256(L.nb * kPieces * L.ntp * kPB);
    L.p_off = L.s_off + round_up_256(L.nb * kPieces * L.ntp);
    L.total = L.p_off + (L.sp.ks > 1 ? round_up_256(4 * L.sp.ks * n_tok * M) : 0);
    return L;
}

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Four threads per (token t, block b): thread q takes elements 4q .. 4q+3
// and 16+4q .. 16+4q+3 of the block, which are fields 8q .. 8q+7 of its
// pieces (field j is element j/2 + 16 (j % 2)); a piece's scale comes from
// the block's largest |r| over the four threads (one lane quad). Thread
// order: q fastest, then the token within its tile, the block, the token
// tile, so that a quad writes one piece's 24 bytes and consecutive quads
// consecutive tokens. The grid covers exactly 4 ntp nb threads.
__global__ void __launch_bounds__(256) xsplit_kernel(const float* __restrict__ x, int64_t N, int64_t K, int64_t nb,
                                                     uint8_t* __restrict__ q, uint8_t* __restrict__ s) {
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int qd = (int)(gid & 3);
    const int64_t u = gid >> 2;
    const int64_t tl = u % kBN, rest = u / kBN;
    const int64_t b = rest % nb, ttile = rest / nb;
    const int64_t t = ttile * kBN + tl;
    float r[8];
    if (t < N) {
        const float* p = x + t * K + 32 * b + 4 * qd;
        const float4 v0 = *reinterpret_cast<const float4*>(p);
        const float4 v1 = *reinterpret_cast<const float4*>(p + 16);
        r[0] = v0.x, r[1] = v1.x, r[2] = v0.y, r[3] = v1.y, r[4] = v0.z, r[5] = v1.z, r[6] = v0.w, r[7] = v1.w;
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) r[k] = 0.f;
    }
#pragma unroll
    for (int pc = 0; pc < kPieces; ++pc) {
        float m = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) m = fmaxf(m, fabsf(r[k]));
        m = fmaxf(m, dpp_move<0xB1>(m));  // quad lanes 1, 0, 3, 2
        m = fmaxf(m, dpp_move<0x4E>(m));  // quad lanes 2, 3, 0, 1
        // m = f 2^e with f in [1/2, 1): floor(log2 m) = e - 1
        int S = m > 0.f ? __builtin_amdgcn_frexp_expf(m) - 2 : -127;
        S = S < -127 ? -127 : S;
        uint64_t w = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float v = __builtin_ldexpf(r[k], -S);  // exact; |v| < 4
            const float a = fabsf(v);
            const bool fine = a < 2.f;  // steps of 1/8 below 2, of 1/4 from 2 to 4
            const float g = __builtin_rintf(a * (fine ? 8.f : 4.f));
            // e2m3 code (sign bit 5, exponent bits 3-4 with bias 1, mantissa
            // bits 0-2): 8a below 2 and 4a + 8 from 2 on are the code's low
            // five bits themselves (subnormals included; 4.0 is code 24)
            const uint32_t code = ((uint32_t)g + (fine ? 0u : 8u)) | (v < 0.f ? 32u : 0u);
            const float qv = g * (fine ? 0.125f : 0.25f);
            r[k] -= __builtin_ldexpf(__builtin_copysignf(qv, v), S);
            w |= (uint64_t)code << (6 * k);
        }
        const int64_t slot = ((ttile * nb + b) * kPieces + pc) * kBN + tl;
        uint16_t* qp = reinterpret_cast<uint16_t*>(q + slot * kPB + 6 * qd);
        qp[0] = (uint16_t)w;
        qp[1] = (uint16_t)(w >> 16);
        qp[2] = (uint16_t)(w >> 32);
        if (qd == 0) s[slot] = (uint8_t)(S + 127);
    }
}

// y[i] = sum over the ks K splits of part[split][i], i < n (float4 where
// n % 4 == 0, whose slices are then 16-byte aligned).
__global__ void __launch_bounds__(256) ksum_kernel(const float* __restrict__ part, int ks, int64_t n,
                                                   float* __restrict__ y) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    const int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if ((n & 3) == 0) {
        const int64_t n4 = n / 4;
        for (int64_t i = i0; i < n4; i += stride) {
            float4 acc = reinterpret_cast<const float4*>(part)[i];
            for (int sp = 1; sp < ks; ++sp) {
                const float4 v = reinterpret_cast<const float4*>(part + sp * n)[i];
                acc.x += v.x, acc.y += v.y, acc.z += v.z, acc.w += v.w;
            }
            reinterpret_cast<float4*>(y)[i] = acc;
        }
    } else {
        for (int64_t i = i0; i < n; i += stride) {
            float acc = part[i];
            for (int sp = 1; sp < ks; ++sp) acc += part[sp * n + i];
            y[i] = acc;
        }
    }
}

template <int NW, int RT>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(RT == 4 ? 1 : 2, RT == 4 ? 1 : 2)))
    fp4mm_kernel(const uint8_t* __restrict__ W, const uint8_t* __restrict__ xq, const uint8_t* __restrict__ xs,
                 float* __restrict__ y, float* __restrict__ part, int64_t M, int64_t K, int64_t N, int64_t off1,
                 GemmSplit sp) {
    constexpr int NT = 64 * NW, BM = 32 * RT * NW;
    constexpr int kChunk = kBN * kPB;                // one (block, piece) of the token tile: 1536 bytes
    constexpr int kStageQ = kSB * kPieces * kChunk;  // codes of a stage
    constexpr int kStageS = kSB * kPieces * kBN;     // scale bytes of a stage
    constexpr int kStage = kStageQ + kStageS;
    constexpr int QU = kStageQ / 16 / NT;  // 16-byte units of codes per thread and stage
    static_assert(QU * 16 * NT == kStageQ, "whole code units per thread");
    constexpr int SB = kStageS / NT;  // scale bytes per thread and stage (2 or 4)
    static_assert(SB * NT == kStageS && (SB == 2 || SB == 4), "whole scale words per thread");
    using SW = typename std::conditional<SB == 4, uint32_t, uint16_t>::type;
    __shared__ __align__(16) uint8_t lds[2 * kStage];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wm = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n32 = lane & 31, h = lane >> 5;

    const int64_t G = (int64_t)gridDim.x;
    const int64_t bi = (int64_t)blockIdx.x;
    const int64_t L = (G & 7) == 0 ? (bi & 7) * (G >> 3) + (bi >> 3) : bi;
    const int64_t tt_i = L % sp.ntt;
    const int64_t rest = L / sp.ntt;
    const int split = (int)(rest % sp.ks);
    const int64_t rti = rest / sp.ks;
    const int64_t row0 = rti * BM;
    const int64_t tok0 = tt_i * kBN;
    const int nsb = (int)(K / 256);
    const int sb0 = split * sp.sbp;
    const int sb1 = sb0 + sp.sbp < nsb ? sb0 + sp.sbp : nsb;
    const int64_t kb0 = 8 * (int64_t)sb0;
    const int nst = 8 * (sb1 - sb0) / kSB;  // at least 1 (every split has a super-block)

    // ---- weights: lane (h, n32) of row tile rt reads row 32 (RT wm + rt) + n32,
    // blocks kWS h .. kWS h + kWS - 1 of each stage and their exponents ----
    const uint8_t* wp[RT];
    const uint8_t* ep[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t r = row0 + 32 * (RT * wm + rt) + n32;
        const int64_t rr = r < M ? r : M - 1;  // past M: a valid row, never stored
        wp[rt] = W + rr * (K / 2) + 16 * (kb0 + kWS * h);
        ep[rt] = W + off1 + rr * (K / 32) + kb0 + kWS * h;
    }
    using EW = typename std::conditional<kWS == 4, uint32_t, uint16_t>::type;
    u32x4v a[2][RT][kWS];  // [buffer][row tile][window]
    uint32_t sa[2][RT];    // the kWS exponent bytes of [buffer][row tile]
    auto load_a = [&](int bf, int st) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const u32x4v* p = reinterpret_cast<const u32x4v*>(wp[rt] + 16 * kSB * (int64_t)st);
#pragma unroll
            for (int j = 0; j < kWS; ++j) a[bf][rt][j] = p[j];
            sa[bf][rt] = *reinterpret_cast<const EW*>(ep[rt] + kSB * (int64_t)st);
        }
    };

    // ---- activation pieces: a stage of the token tile is kStageQ contiguous
    // bytes of codes (chunk c = 4 b + p: block b of the stage, piece p, 64
    // tokens) and kStageS of scales, copied to LDS in 16-byte units ----
    const int64_t nb = K / 32;
    const uint8_t* qsrc = xq + ((tt_i * nb + kb0) * kPieces * kBN) * kPB + 16 * tid;
    const uint8_t* ssrc = xs + (tt_i * nb + kb0) * kPieces * kBN + SB * tid;
    u32x4v qreg[QU];
    SW sreg;
    auto fetch = [&](int st) __attribute__((always_inline)) {
        const uint8_t* q = qsrc + (int64_t)kStageQ * st;
#pragma unroll
        for (int i = 0; i < QU; ++i) qreg[i] = *reinterpret_cast<const u32x4v*>(q + 16 * NT * i);
        sreg = *reinterpret_cast<const SW*>(ssrc + (int64_t)kStageS * st);
    };
    auto commit = [&](int bf) __attribute__((always_inline)) {
        uint8_t* base = lds + bf * kStage + 16 * tid;
#pragma unroll
        for (int i = 0; i < QU; ++i) *reinterpret_cast<u32x4v*>(base + 16 * NT * i) = qreg[i];
        *reinterpret_cast<SW*>(lds + bf * kStage + kStageQ + SB * tid) = sreg;
    };

    f32x16 acc[RT][2];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[rt][tt][v] = 0.f;

    // B operands (pieces) and their scales of group g = 4 j + p (window j,
    // piece p) for both token tiles, read from LDS one group ahead of the
    // group's MFMAs; the scheduling barriers keep the compiler from hoisting
    // every group's reads to the top (which would hold all of them in
    // registers at once)
    struct BOps {
        i32x8 op[2];
        int sc[2];
    };
    auto read_b = [&](int bf, int g) __attribute__((always_inline)) {
        const uint8_t* base = lds + bf * kStage;
        const int j = g / kPieces, pc = g % kPieces;
        const int c = (kWS * h + j) * kPieces + pc;  // this lane half's block of window j
        BOps b;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
            const uint2* p = reinterpret_cast<const uint2*>(base + c * kChunk + (32 * tt + n32) * kPB);
            const uint2 v0 = p[0], v1 = p[1], v2 = p[2];
            b.op[tt] = i32x8{(int)v0.x, (int)v0.y, (int)v1.x, (int)v1.y, (int)v2.x, (int)v2.y, 0, 0};
            b.sc[tt] = base[kStageQ + c * kBN + 32 * tt + n32];
        }
        return b;
    };
    auto compute = [&](int bf) __attribute__((always_inline)) {
        BOps nxt = read_b(bf, 0);
#pragma unroll
        for (int g = 0; g < kWS * kPieces; ++g) {
            const BOps cur = nxt;
            if (g + 1 < kWS * kPieces) nxt = read_b(bf, g + 1);
            const int j = g / kPieces;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const u32x4v av = a[bf][rt][j];
                const i32x8 aop = {(int)av[0], (int)av[1], (int)av[2], (int)av[3], 0, 0, 0, 0};
                const int sav = (int)((sa[bf][rt] >> (8 * j)) & 0xFFu);
#pragma unroll
                for (int tt = 0; tt < 2; ++tt)
                    acc[rt][tt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(aop, cur.op[tt], acc[rt][tt], 4, 2, 0,
                                                                                  sav, 0, cur.sc[tt]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // ---- prologue: stage 0 in LDS buffer 0 and registers a[0]; stage 1 (or a
    // copy of the last) in flight. Loads past the split's end are clamped to
    // its last stage: valid addresses whose values are never used ----
    load_a(0, 0);
    fetch(0);
    commit(0);
    load_a(1, nst > 1 ? 1 : 0);
    fetch(nst > 1 ? 1 : 0);
    __syncthreads();
    // stages in pairs, so that every register buffer index is a constant: LDS
    // buffer and a[] buffer b hold the stages of parity b (an odd count ends
    // after the first of its last pair)
    for (int st = 0; st < nst; st += 2) {
        const int s2 = st + 2 < nst ? st + 2 : nst - 1, s3 = st + 3 < nst ? st + 3 : nst - 1;
        commit(1);  // stage st + 1
        fetch(s2);
        compute(0);
        load_a(0, s2);
        __syncthreads();
        if (st + 1 == nst) break;
        commit(0);  // stage st + 2 (past the end: a copy of the last, never read)
        fetch(s3);
        compute(1);
        load_a(1, s3);
        __syncthreads();
    }

    // store: lane (h, n32) holds token 32 tt + n32 of rows 32 (RT wm + rt) +
    // 8 g + 4 h + e (register 4 g + e); a K split writes its own slice of
    // the partial results (part), summed into y afterwards
    float* const out = sp.ks > 1 ? part + (int64_t)split * N * M : y;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
        const int64_t t = tok0 + 32 * tt + n32;
        if (t >= N) continue;
        float* const yt = out + t * M;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int64_t r = row0 + 32 * (RT * wm + rt) + 8 * g + 4 * h;
                const f32x16& v = acc[rt][tt];
                if ((M & 3) == 0 && r + 3 < M) {
                    *reinterpret_cast<float4*>(yt + r) = make_float4(v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (r + e < M) yt[r + e] = v[4 * g + e];
                }
            }
    }
}

}  // namespace

bool fp4mm_takes(int fmt, int64_t n_tok) { return fmt == LW_MXFP4 && n_tok > 16; }

int64_t fp4mm_workspace_bytes(int64_t M, int64_t K, int64_t n_tok) { return xlayout(M, K, n_tok).total; }

hipError_t launch_fp4mm(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                        const Planes& p, uint8_t* ws, hipStream_t stream) {
    const XLayout L = xlayout(M, K, n_tok);
    const GemmSplit& sp = L.sp;
    const int64_t grid = sp.nrt * sp.ntt * sp.ks;
    const int64_t sgrid = 4 * L.ntp * L.nb / 256;  // ntp is a multiple of 64: whole workgroups
    const int64_t n = n_tok * M;
    const int64_t rgrid = (n / 4 + 255) / 256 < 4096 ? (n / 4 + 255) / 256 + 1 : 4096;
    if (grid > 0x7fffffff || sgrid > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (query_only(kernel_name<Name_fp4mm_kernel, kNW, kRT>(), sp.ks > 1 ? 3 : 2)) return hipSuccess;
    hipLaunchKernelGGL(xsplit_kernel, dim3((unsigned)sgrid), dim3(256), 0, stream, x, n_tok, K, L.nb, ws, ws + L.s_off);
    float* part = reinterpret_cast<float*>(ws + L.p_off);
    hipLaunchKernelGGL((fp4mm_kernel<kNW, kRT>), dim3((unsigned)grid), dim3(64 * kNW), 0, stream, W, ws,
                       ws + L.s_off, y, part, M, K, n_tok, p.off1, sp);
    if (sp.ks > 1)
        hipLaunchKernelGGL(ksum_kernel, dim3((unsigned)rgrid), dim3(256), 0, stream, part, sp.ks, n, y);
    return hipGetLastError();
}

}  // namespace lw
