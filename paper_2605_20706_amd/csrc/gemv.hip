// Fused dequantize x matrix-vector product (decode, n_tok <= LW_GEMV_MAX_TOK).
//
// y[t][r] = sum_k value(W, r*K + k) * x[t][k]  (Sec. 2.1: decode is a
// matrix-vector product; Sec. 3.3: the matrix-vector kernel dequantizes the
// weights directly into registers instead of tiling them through shared
// memory, and the vector is tiled and the row reduced cooperatively, Sec. 3.2).
//
// Mapping on gfx950 (wave64):
//  * A chunk is 64 lanes x 16 bytes = 1 KiB of a row's code plane: 2048
//    elements for the 4-bit formats, 1024 for Q8_0, 512 for f16. Lane l loads
//    its 16 bytes with one 128-bit load, so each wave-wide load is one
//    contiguous KiB; its block scale(s) are loaded beside it.
//  * Each wave owns R consecutive rows and walks their chunks, keeping R x NT
//    float32 partial sums per lane; at the end the 64 lanes are summed with
//    DPP adds and lane 63 stores the R x NT results.
//  * The workgroup stages its x tile once in LDS in a lane-interleaved order
//    (float4 j of lane l of chunk c at index (c*J + j)*64 + l), so every
//    128-bit LDS read of a wave is 64 consecutive float4s (no bank conflicts);
//    one x read serves the R rows of the wave.
//  * Codes become floats with one v_cvt_f32_ubyteN each (4-bit: the low and
//    high nibbles are masked in place, the high-nibble sum is scaled by 1/16
//    at the end); block scales are applied once per 32 elements in factored
//    form: Q4_0 d*(sum q*x - 8*sum x), Q4_K-style d*sc*sum q*x - dmin*m*sum x,
//    with the per-group sums of x precomputed in LDS per tile.
// Accumulation is float32 throughout; only the rounding order differs from
// the plain definition.
#include <atomic>

#include "lw_device.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

constexpr int64_t kLdsBytes = 64 * 1024;  // LDS budget of a workgroup (x tile + group sums)

template <int FMT>
struct Traits;

template <>
struct Traits<LW_F16> {
    static constexpr int EPL = 8;  // elements per lane per chunk
    static constexpr bool kGroupSums = false;
    struct Packet {
        uint4 c;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t, int64_t) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + 2 * e);
        return p;
    }
    // Byte offsets of row `row` in each plane, lane part included (32-bit:
    // the kernel using them is chosen only for planes below 4 GiB), and the
    // packet of chunk c (512 elements) at those offsets.
    struct RowOff {
        uint32_t c;
    };
    __device__ static RowOff row_off(uint32_t row, uint32_t K, int lane) { return {row * (2u * K) + 16u * lane}; }
    __device__ static Packet load_chunk(const uint8_t* W, const uint8_t*, const uint8_t*, const RowOff& o, int c) {
        Packet p;
        p.c = stream_load16(W + (o.c + 1024u * c));
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float, int) {
        float s = 0.f;
        s = __builtin_fmaf(half_bits_to_float(p.c.x & 0xFFFFu), xv[0].x, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.x >> 16), xv[0].y, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.y & 0xFFFFu), xv[0].z, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.y >> 16), xv[0].w, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.z & 0xFFFFu), xv[1].x, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.z >> 16), xv[1].y, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.w & 0xFFFFu), xv[1].z, s);
        s = __builtin_fmaf(half_bits_to_float(p.c.w >> 16), xv[1].w, s);
        return s;
    }
};

template <>
struct Traits<LW_Q8_0> {
    static constexpr int EPL = 16;
    static constexpr bool kGroupSums = false;
    struct Packet {
        uint4 c;
        uint32_t d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + e);
        p.d = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 5));
        return p;
    }
    struct RowOff {
        uint32_t c, d;
    };
    __device__ static RowOff row_off(uint32_t row, uint32_t K, int lane) {
        return {row * K + 16u * lane, row * (K / 16u) + 2u * (lane >> 1)};
    }
    __device__ static Packet load_chunk(const uint8_t* W, const uint8_t* P1, const uint8_t*, const RowOff& o,
                                        int c) {  // chunk = 1024 elements
        Packet p;
        p.c = stream_load16(W + (o.c + 1024u * c));
        p.d = *reinterpret_cast<const uint16_t*>(P1 + (o.d + 64u * c));
        return p;
    }
    __device__ static float dot(const Packet& p, const float4* xv, float, int) {
        const uint32_t w[4] = {p.c.x, p.c.y, p.c.z, p.c.w};
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            s0 = __builtin_fmaf(sbyte<0>(w[i]), xv[i].x, s0);
            s1 = __builtin_fmaf(sbyte<1>(w[i]), xv[i].y, s1);
            s0 = __builtin_fmaf(sbyte<2>(w[i]), xv[i].z, s0);
            s1 = __builtin_fmaf(sbyte<3>(w[i]), xv[i].w, s1);
        }
        return half_bits_to_float(p.d) * (s0 + s1);
    }
};

// Sum over the lane's 32 elements of q * x for 4-bit codes: returns
// sum_lo + sum_hi / 16, where the high nibbles are converted in place as 16*q.
__device__ __forceinline__ float nibble_dot(const uint4& c, const float4* xv) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    float lo_s = 0.f, hi_s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t lo = opaque(w[i] & 0x0F0F0F0Fu);  // elements 4i .. 4i+3
        const uint32_t hi = opaque(w[i] & 0xF0F0F0F0u);  // elements 16+4i .. 16+4i+3, times 16
        lo_s = __builtin_fmaf(ubyte<0>(lo), xv[i].x, lo_s);
        lo_s = __builtin_fmaf(ubyte<1>(lo), xv[i].y, lo_s);
        lo_s = __builtin_fmaf(ubyte<2>(lo), xv[i].z, lo_s);
        lo_s = __builtin_fmaf(ubyte<3>(lo), xv[i].w, lo_s);
        hi_s = __builtin_fmaf(ubyte<0>(hi), xv[4 + i].x, hi_s);
        hi_s = __builtin_fmaf(ubyte<1>(hi), xv[4 + i].y, hi_s);
        hi_s = __builtin_fmaf(ubyte<2>(hi), xv[4 + i].z, hi_s);
        hi_s = __builtin_fmaf(ubyte<3>(hi), xv[4 + i].w, hi_s);
    }
    return __builtin_fmaf(hi_s, 0.0625f, lo_s);
}

template <>
struct Traits<LW_Q4_0> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t d;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        p.d = *reinterpret_cast<const uint16_t*>(W + off1 + 2 * (e >> 5));
        return p;
    }
    struct RowOff {
        uint32_t c, d;
    };
    __device__ static RowOff row_off(uint32_t row, uint32_t K, int lane) {
        return {row * (K / 2u) + 16u * lane, row * (K / 16u) + 2u * lane};
    }
    __device__ static Packet load_chunk(const uint8_t* W, const uint8_t* P1, const uint8_t*, const RowOff& o,
                                        int c) {  // chunk = 2048 elements
        Packet p;
        p.c = stream_load16(W + (o.c + 1024u * c));
        p.d = *reinterpret_cast<const uint16_t*>(P1 + (o.d + 128u * c));
        return p;
    }
    // d * (sum q*x - 8 * sum x)
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int) {
        return half_bits_to_float(p.d) * __builtin_fmaf(-8.0f, sx, nibble_dot(p.c, xv));
    }
};

template <>
struct Traits<LW_Q4_K> {
    static constexpr int EPL = 32;
    static constexpr bool kGroupSums = true;
    struct Packet {
        uint4 c;
        uint32_t r0, r1, r2, dd;
    };
    __device__ static Packet load(const uint8_t* W, int64_t e, int64_t off1, int64_t off2) {
        Packet p;
        p.c = *reinterpret_cast<const uint4*>(W + (e >> 1));
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(W + off1 + 12 * (e >> 8));
        p.r0 = rec[0];
        p.r1 = rec[1];
        p.r2 = rec[2];
        p.dd = *reinterpret_cast<const uint32_t*>(W + off2 + 4 * (e >> 8));
        return p;
    }
    struct RowOff {
        uint32_t c, rec, dd;
    };
    __device__ static RowOff row_off(uint32_t row, uint32_t K, int lane) {
        return {row * (K / 2u) + 16u * lane, row * (12u * (K / 256u)) + 12u * (lane >> 3),
                row * (4u * (K / 256u)) + 4u * (lane >> 3)};
    }
    __device__ static Packet load_chunk(const uint8_t* W, const uint8_t* P1, const uint8_t* P2, const RowOff& o,
                                        int c) {  // chunk = 2048 elements = 8 super-blocks
        Packet p;
        p.c = stream_load16(W + (o.c + 1024u * c));
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(P1 + (o.rec + 96u * c));
        p.r0 = rec[0];
        p.r1 = rec[1];
        p.r2 = rec[2];
        p.dd = *reinterpret_cast<const uint32_t*>(P2 + (o.dd + 32u * c));
        return p;
    }
    // d*sc_j * sum q*x - dmin*m_j * sum x; j is the lane's sub-block (0..7).
    __device__ static float dot(const Packet& p, const float4* xv, float sx, int j) {
        const uint64_t lo = (uint64_t)p.r0 | ((uint64_t)p.r1 << 32);  // record bits 0..63
        const uint64_t hi = (uint64_t)p.r1 | ((uint64_t)p.r2 << 32);  // record bits 32..95
        const float sc = (float)((uint32_t)(lo >> (6 * j)) & 63u);
        const float m = (float)((uint32_t)(hi >> (16 + 6 * j)) & 63u);
        const float ds = half_bits_to_float(p.dd & 0xFFFFu) * sc;
        const float dm = half_bits_to_float(p.dd >> 16) * m;
        return __builtin_fmaf(ds, nibble_dot(p.c, xv), -dm * sx);
    }
};

template <int FMT, int NT, int R, int NW>
__global__ void __launch_bounds__(NW * kWave)
    gemv_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y,
                int64_t M, int64_t K, int KT, int64_t off1, int64_t off2) {
    using T = Traits<FMT>;
    constexpr int EPL = T::EPL;
    constexpr int J4 = EPL / 4;  // float4s of x per lane per chunk
    constexpr int E = kWave * EPL;
    extern __shared__ float4 smem[];

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t row_base = ((int64_t)blockIdx.x * NW + wave) * R;
    if (KT <= 0) return;               // never launched so; keeps the tile loop finite
    const int nch = (KT + E - 1) / E;  // chunks in a full tile
    const int tok4 = nch * E / 4;      // float4s per token in the LDS tile
    float4* xs = smem;
    float* sxs = reinterpret_cast<float*>(smem + NT * tok4);  // [NT][nch * 64] group sums

    int64_t rows[R];
#pragma unroll
    for (int r = 0; r < R; ++r) rows[r] = (row_base + r < M) ? row_base + r : M - 1;

    float acc[R][NT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[r][t] = 0.f;

    for (int64_t k0 = 0; k0 < K; k0 += KT) {
        const int kt = (int)((K - k0) < KT ? (K - k0) : KT);
        if (k0) __syncthreads();  // every wave is done with the previous tile
        // Stage x[:, k0 : k0+kt] (coalesced global reads, lane-interleaved LDS order).
        const int n4 = kt / 4;
        for (int idx = threadIdx.x; idx < NT * n4; idx += NW * kWave) {
            const int t = idx / n4, q = idx - t * n4;
            const int k = 4 * q;
            const int c = k / E, w = k - c * E, l = w / EPL, j4 = (w - l * EPL) / 4;
            xs[t * tok4 + (c * J4 + j4) * kWave + l] =
                *reinterpret_cast<const float4*>(x + (int64_t)t * K + k0 + k);
        }
        __syncthreads();
        if constexpr (T::kGroupSums) {
            const int ng = kt / 32;
            for (int idx = threadIdx.x; idx < NT * ng; idx += NW * kWave) {
                const int t = idx / ng, g = idx - t * ng;
                const int c = g / kWave, l = g - c * kWave;
                float s = 0.f;
#pragma unroll
                for (int j4 = 0; j4 < 8; ++j4) {
                    const float4 v = xs[t * tok4 + (c * 8 + j4) * kWave + l];
                    s += (v.x + v.y) + (v.z + v.w);
                }
                sxs[t * nch * kWave + g] = s;
            }
            __syncthreads();
        }

        const int nc = (kt + E - 1) / E;
        for (int c = 0; c < nc; ++c) {
            const int kl = c * E + lane * EPL;  // first element of the lane, within the tile
            if (kl < kt) {
                const int64_t kk = k0 + kl;
                typename T::Packet pk[R];
#pragma unroll
                for (int r = 0; r < R; ++r) pk[r] = T::load(W, rows[r] * K + kk, off1, off2);
                const int j = (int)((kk >> 5) & 7);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    float4 xv[J4];
#pragma unroll
                    for (int j4 = 0; j4 < J4; ++j4) xv[j4] = xs[t * tok4 + (c * J4 + j4) * kWave + lane];
                    const float sx = T::kGroupSums ? sxs[t * nch * kWave + c * kWave + lane] : 0.f;
#pragma unroll
                    for (int r = 0; r < R; ++r) acc[r][t] += T::dot(pk[r], xv, sx, j);
                }
            }
        }
    }

#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float v = wave_sum_to_lane63(acc[r][t]);
            if (lane == kWave - 1 && row_base + r < M) y[(int64_t)t * M + row_base + r] = v;
        }
}

// Single-token kernel. The workgroup is persistent: it stages x once and then
// walks row batches (R rows) with a stride of the whole grid. A batch is split
// into steps of CH chunks; each wave keeps the packets of its next step in
// flight while it computes the current one. To keep the start short, every
// thread first issues its x loads, then the loads of its first step, and only
// then waits for x (vector-memory results return in issue order), so the x
// tile and its group sums are in LDS after one barrier while the weights are
// still on their way.
template <int FMT, int R, int CH, int NW>
__global__ void __launch_bounds__(NW * kWave)
    gemv1_kernel(const uint8_t* __restrict__ W, const float* __restrict__ x, float* __restrict__ y,
                 int64_t M, int64_t K, int64_t off1, int64_t off2) {
    using T = Traits<FMT>;
    constexpr int EPL = T::EPL;
    constexpr int J4 = EPL / 4;
    constexpr int E = kWave * EPL;
    extern __shared__ float4 smem[];

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int nc = (int)((K + E - 1) / E);  // chunks per row
    const int ns = (nc + CH - 1) / CH;      // steps per row batch
    float4* xs = smem;                                          // nc * E floats, lane-interleaved
    float* sxs = reinterpret_cast<float*>(smem + nc * (E / 4));  // nc * 64 group sums (4-bit formats)
    const int64_t nbatch = (M + R - 1) / R;
    const int64_t bstride = (int64_t)gridDim.x * NW;
    int64_t b = (int64_t)blockIdx.x * NW + wave;

    // (1) x loads first: thread t owns lane-slices t, t + blockDim, ... (EPL floats each).
    const int nsl = (int)(K / EPL);
    const int t0 = threadIdx.x;
    float4 xr[J4];
    if (t0 < nsl) {
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) xr[j4] = *reinterpret_cast<const float4*>(x + (int64_t)EPL * t0 + 4 * j4);
    }

    // (2) the first step of this wave's first batch. Row offsets (32-bit,
    // plane bases uniform) are formed once per batch, not per step.
    const uint32_t K32 = (uint32_t)K;
    const uint8_t* P1 = W + off1;
    const uint8_t* P2 = W + off2;
    typename T::Packet cur[R][CH], nxt[R][CH];
    typename T::RowOff ro[R];  // rows of the batch whose steps are being issued
    auto row_offs = [&](int64_t bb) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t rr = bb * R + r;
            ro[r] = T::row_off((uint32_t)(rr < M ? rr : M - 1), K32, lane);
        }
    };
    auto load_step = [&](typename T::Packet (*pk)[CH], int ss) {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int cc = 0; cc < CH; ++cc) {
                const int c = ss * CH + cc;
                if ((uint32_t)(c * E + lane * EPL) < K32) pk[r][cc] = T::load_chunk(W, P1, P2, ro[r], c);
            }
    };
    if (b < nbatch) {
        row_offs(b);
        load_step(cur, 0);
    }

    // (3) x into LDS (and the group sums), one barrier
    auto put_slice = [&](int t, const float4* v) {
        const int c = t / kWave, l = t - c * kWave;
        float sum = 0.f;
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) {
            xs[(c * J4 + j4) * kWave + l] = v[j4];
            sum += (v[j4].x + v[j4].y) + (v[j4].z + v[j4].w);
        }
        if (T::kGroupSums) sxs[t] = sum;
    };
    if (t0 < nsl) put_slice(t0, xr);
    for (int t = t0 + NW * kWave; t < nsl; t += NW * kWave) {
        float4 v[J4];
#pragma unroll
        for (int j4 = 0; j4 < J4; ++j4) v[j4] = *reinterpret_cast<const float4*>(x + (int64_t)EPL * t + 4 * j4);
        put_slice(t, v);
    }
    __syncthreads();

    // (4) stream the batches
    const int j = lane & 7;
    int s = 0;
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
    while (b < nbatch) {
        int64_t nb = b;
        int nss = s + 1;
        if (nss == ns) {
            nss = 0;
            nb += bstride;
        }
        if (nb < nbatch) {
            // every step of batch b is already issued when the next batch starts
            if (nss == 0) row_offs(nb);
            load_step(nxt, nss);
        }
#pragma unroll
        for (int cc = 0; cc < CH; ++cc) {
            const int c = s * CH + cc;
            if ((uint32_t)(c * E + lane * EPL) < K32) {
                float4 xv[J4];
#pragma unroll
                for (int j4 = 0; j4 < J4; ++j4) xv[j4] = xs[(c * J4 + j4) * kWave + lane];
                const float sx = T::kGroupSums ? sxs[c * kWave + lane] : 0.f;
#pragma unroll
                for (int r = 0; r < R; ++r) acc[r] += T::dot(cur[r][cc], xv, sx, j);
            }
        }
        if (s == ns - 1) {
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const float v = wave_sum_to_lane63(acc[r]);
                if (lane == kWave - 1 && b * R + r < M) y[b * R + r] = v;
                acc[r] = 0.f;
            }
        }
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int cc = 0; cc < CH; ++cc) cur[r][cc] = nxt[r][cc];
        b = nb;
        s = nss;
    }
}

struct Config {
    int R, NW;
};

template <int FMT, int NT>
hipError_t launch_nt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                     const Planes& p, hipStream_t stream) {
    constexpr int E = kWave * Traits<FMT>::EPL;
    constexpr int R = NT == 1 ? 4 : (NT <= 4 ? 2 : 1);
    constexpr int NW = 4;
    // x tile: the whole K if it fits the LDS budget, else the largest whole
    // number of chunks that does (each chunk: NT x E floats of x, plus NT x 64
    // group sums for the 4-bit formats).
    const int64_t chunk_bytes = (int64_t)NT * (E * 4 + (Traits<FMT>::kGroupSums ? kWave * 4 : 0));
    int64_t nch = (K + E - 1) / E;
    if (nch * chunk_bytes > kLdsBytes) nch = kLdsBytes / chunk_bytes;
    if (nch < 1) return hipErrorInvalidConfiguration;  // callers split tokens first (see fits_one_chunk)
    const int64_t KT = nch * E;
    const size_t lds = (size_t)(nch * chunk_bytes);
    const int64_t blocks = (M + (int64_t)NW * R - 1) / ((int64_t)NW * R);
    hipLaunchKernelGGL((gemv_kernel<FMT, NT, R, NW>), dim3((unsigned)blocks), dim3(NW * kWave), lds,
                       stream, W, x, y, M, K, (int)KT, p.off1, p.off2);
    return hipGetLastError();
}

// Whether one chunk of x for NT tokens (plus its group sums) fits the LDS budget.
template <int FMT, int NT>
constexpr bool fits_one_chunk() {
    return (int64_t)NT * (kWave * Traits<FMT>::EPL * 4 + (Traits<FMT>::kGroupSums ? kWave * 4 : 0)) <=
           kLdsBytes;
}

// Compute units of the current device, looked up once per device.
int cu_count() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v <= 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// Single token: the persistent kernel when the whole x row fits the LDS
// budget, else the K-tiled kernel.
template <int FMT, int R, int CH>
hipError_t launch_single(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                         const Planes& p, hipStream_t stream) {
    constexpr int NW = 8;
    constexpr int E = kWave * Traits<FMT>::EPL;
    const int64_t nc = (K + E - 1) / E;
    const int64_t lds = nc * E * 4 + (Traits<FMT>::kGroupSums ? nc * kWave * 4 : 0);
    if (lds > kLdsBytes || p.total >= ((int64_t)1 << 32) || M >= ((int64_t)1 << 31))
        return launch_nt<FMT, 1>(W, x, y, M, K, p, stream);
    const int64_t nbatch = (M + R - 1) / R;
    int64_t grid = (nbatch + NW - 1) / NW;
    const int64_t cap = 2 * (int64_t)cu_count();  // two 8-wave workgroups per CU
    if (grid > cap) grid = cap;
    hipLaunchKernelGGL((gemv1_kernel<FMT, R, CH, NW>), dim3((unsigned)grid), dim3(NW * kWave), (size_t)lds,
                       stream, W, x, y, M, K, p.off1, p.off2);
    return hipGetLastError();
}

template <int FMT>
hipError_t launch_fmt(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                      int64_t n_tok, const Planes& p, hipStream_t stream) {
    if (n_tok == 1) {
        if constexpr (FMT == LW_Q4_0) return launch_single<FMT, 4, 1>(W, x, y, M, K, p, stream);

        return launch_single<FMT, 2, 1>(W, x, y, M, K, p, stream);
    }
    if constexpr (!fits_one_chunk<FMT, 8>()) {
        // 8 tokens of a 4-bit chunk (64 KiB of x) plus group sums exceed the
        // budget: run them as two launches of 4 tokens.
        if (n_tok == 8) {
            hipError_t err = launch_nt<FMT, 4>(W, x, y, M, K, p, stream);
            if (err != hipSuccess) return err;
            return launch_nt<FMT, 4>(W, x + 4 * K, y + 4 * M, M, K, p, stream);
        }
    }
    switch (n_tok) {
    case 1: return launch_nt<FMT, 1>(W, x, y, M, K, p, stream);
    case 2: return launch_nt<FMT, 2>(W, x, y, M, K, p, stream);
    case 3: return launch_nt<FMT, 3>(W, x, y, M, K, p, stream);
    case 4: return launch_nt<FMT, 4>(W, x, y, M, K, p, stream);
    case 5: return launch_nt<FMT, 5>(W, x, y, M, K, p, stream);
    case 6: return launch_nt<FMT, 6>(W, x, y, M, K, p, stream);
    case 7: return launch_nt<FMT, 7>(W, x, y, M, K, p, stream);
    case 8:
        if constexpr (fits_one_chunk<FMT, 8>()) return launch_nt<FMT, 8>(W, x, y, M, K, p, stream);
        return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_gemv(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                       int64_t n_tok, const Planes& p, hipStream_t stream) {
    switch (fmt) {
    case LW_F16: return launch_fmt<LW_F16>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q8_0: return launch_fmt<LW_Q8_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_0: return launch_fmt<LW_Q4_0>(W, x, y, M, K, n_tok, p, stream);
    case LW_Q4_K: return launch_fmt<LW_Q4_K>(W, x, y, M, K, n_tok, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
