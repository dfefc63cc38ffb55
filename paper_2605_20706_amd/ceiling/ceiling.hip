// Streaming ceilings: a plain 128-bit read and a plain 128-bit non-temporal
// write of a buffer, timed by the benchmark beside the product kernels (the
// rate they reach bounds any kernel that moves the same bytes).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "lw_ceiling.h"

namespace {

// One 512-thread workgroup per compute unit, four 16-byte non-temporal loads
// in flight per thread: the fastest plain read form in a sweep of grid and
// workgroup sizes on MI355X (6.9 TB/s over 295 MB per launch).
constexpr int kThreads = 512;
constexpr int kUnroll = 4;

__global__ void __launch_bounds__(kThreads) read_kernel(const uint4* __restrict__ p, int64_t n16,
                                                        uint32_t* __restrict__ sink) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(q + i + u * stride);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc ^= v[u];
    }
    for (; i < n16; i += stride) acc ^= q[i];
    const uint32_t r = acc.x ^ acc.y ^ acc.z ^ acc.w;
    if (r == 0x9E3779B9u) sink[0] = r;
}

__global__ void __launch_bounds__(kThreads) write_kernel(float4* __restrict__ p, int64_t n16) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += stride)
        __builtin_nontemporal_store(f32x4{0.f, 0.f, 0.f, 0.f}, reinterpret_cast<f32x4*>(p + i));
}

// one workgroup per compute unit (fewer for small buffers)
unsigned grid_for(int64_t n16) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    int64_t g = (n16 + (int64_t)kThreads * kUnroll - 1) / ((int64_t)kThreads * kUnroll);
    if (g > cus) g = cus;
    return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

extern "C" int lw_ceiling_read(const void* p, int64_t bytes, uint32_t* sink, void* stream) {
    if (!p || !sink || bytes <= 0 || bytes % 16 || reinterpret_cast<uintptr_t>(p) % 16) return -1;
    const int64_t n16 = bytes / 16;
    hipLaunchKernelGGL(read_kernel, dim3(grid_for(n16)), dim3(kThreads), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint4*>(p), n16, sink);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

extern "C" int lw_ceiling_write(void* p, int64_t bytes, void* stream) {
    if (!p || bytes <= 0 || bytes % 16 || reinterpret_cast<uintptr_t>(p) % 16) return -1;
    const int64_t n16 = bytes / 16;
    hipLaunchKernelGGL(write_kernel, dim3(grid_for(n16)), dim3(kThreads), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<float4*>(p), n16);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}
