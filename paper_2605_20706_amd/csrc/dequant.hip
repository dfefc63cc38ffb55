// Standalone dequantization: packed split-plane weights -> float32, bit-exact.
//
// Each element's closed form (Eq. (1) of Sec. 2.2 with the legacy and K-quant
// block structures of Sec. 2.2) is evaluated with exact float32 products and at
// most one rounding: q*d and (q-8)*d are exact products; the K-quant style
// value d*sc*q - dmin*m (Q4_K-, Q5_K-, Q2_K-style) is one fused
// multiply-add of the exact d*sc and the exact dmin*m, and Q4_1's and Q5_1's
// q*d + m one fused multiply-add of the exact q*d and m; Q6_K-style
// d*sc*(q - 32) is exact (at most 23 significant bits). No half-precision
// arithmetic is used.
//
// Work split: per grid-stride step a thread writes four float4 (4 consecutive
// elements each), 256 float4 apart, so each store instruction of a wave is
// one contiguous 1 KiB; all four values are computed before any is stored,
// which keeps four loads of each kind in flight. The op is bound by the
// float32 writes (4 bytes out per 0.56-2 bytes in). They are non-temporal:
// the output is written once and is far larger than the caches (15-20 %
// faster than plain stores on MI355X).
#include "lw_device.hpp"
#include "lw_formats.hpp"
#include "lw_internal.hpp"

namespace lw {
namespace {

// names of the kernel templates, for lw_kernel_name
struct Name_dequant_kernel {
    static constexpr const char* base = "dequant_kernel";
};

constexpr int kDqU = 4;  // float4 per thread and grid-stride step

template <int FMT>
__global__ void __launch_bounds__(256) dequant_kernel(const uint8_t* __restrict__ W,
                                                      float4* __restrict__ out, int64_t n4,
                                                      int64_t off1, int64_t off2, int64_t off3) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * kDqU;
    for (int64_t base = (int64_t)blockIdx.x * blockDim.x * kDqU + threadIdx.x; base < n4; base += stride) {
        float4 v[kDqU];
#pragma unroll
        for (int u = 0; u < kDqU; ++u) {
            const int64_t i = base + (int64_t)u * blockDim.x;
            v[u] = value4<FMT>(W, off1, off2, off3, 4 * (i < n4 ? i : n4 - 1));  // past the end: a copy, not stored
        }
#pragma unroll
        for (int u = 0; u < kDqU; ++u) {
            const int64_t i = base + (int64_t)u * blockDim.x;
            if (i < n4)
                __builtin_nontemporal_store(f32x4{v[u].x, v[u].y, v[u].z, v[u].w}, reinterpret_cast<f32x4*>(out + i));
        }
    }
}

template <int FMT>
hipError_t launch(const uint8_t* W, float* out, int64_t n, const Planes& p, hipStream_t stream) {
    const int64_t n4 = n / 4;
    const int threads = 256;
    int64_t blocks = (n4 + threads * kDqU - 1) / (threads * kDqU);
    const int64_t cap = 256 * 32;  // 32 workgroups per CU on 256 CUs; the rest is grid-stride
    if (blocks > cap) blocks = cap;
    if (query_only(kernel_name<Name_dequant_kernel, FMT>())) return hipSuccess;
    hipLaunchKernelGGL(dequant_kernel<FMT>, dim3((unsigned)blocks), dim3(threads), 0, stream, W,
                       reinterpret_cast<float4*>(out), n4, p.off1, p.off2, p.off3);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_dequant(int fmt, const uint8_t* W, float* out, int64_t n, const Planes& p,
                          hipStream_t stream) {
    switch (fmt) {
    case LW_F16: return launch<LW_F16>(W, out, n, p, stream);
    case LW_Q8_0: return launch<LW_Q8_0>(W, out, n, p, stream);
    case LW_Q4_0: return launch<LW_Q4_0>(W, out, n, p, stream);
    case LW_Q4_K: return launch<LW_Q4_K>(W, out, n, p, stream);
    case LW_Q4_1: return launch<LW_Q4_1>(W, out, n, p, stream);
    case LW_Q1_0: return launch<LW_Q1_0>(W, out, n, p, stream);
    case LW_Q5_0: return launch<LW_Q5_0>(W, out, n, p, stream);
    case LW_Q5_1: return launch<LW_Q5_1>(W, out, n, p, stream);
    case LW_Q5_K: return launch<LW_Q5_K>(W, out, n, p, stream);
    case LW_Q6_K: return launch<LW_Q6_K>(W, out, n, p, stream);
    case LW_Q2_K: return launch<LW_Q2_K>(W, out, n, p, stream);
    case LW_MXFP4: return launch<LW_MXFP4>(W, out, n, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace lw
