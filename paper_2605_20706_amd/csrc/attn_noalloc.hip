// lw_attn_decode_noalloc: lw_attn_decode for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops). The
// partial results that lw_attn_decode keeps in a caller-provided workspace
// live here in a file-scope device array of kAttnScratchBytes, one per GPU,
// held until the process ends.
//
// The array's name denotes a host-side stand-in in host code, not a device
// address: its device address is taken with hipGetSymbolAddress once per
// device (with that device current, on the first call there) and only that
// address is passed to the kernels. Every call on a GPU shares the GPU's
// array, so calls that overlap in time on one GPU race; the kernels write
// every partial they read within a call, so nothing needs clearing.
#include <atomic>
#include <mutex>

#include "lw_internal.hpp"

namespace {

constexpr int64_t kAttnScratchBytes = 2 << 20;  // 2 MiB per GPU
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kAttnScratchBytes];

std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of this device's scratch array, looked up once per device
// with the device current; nullptr when the lookup fails.
void* scratch_ptr(int dev) {
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p) return p;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
        void* addr = nullptr;
        if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return nullptr;
        p = addr;
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    return p;
}

}  // namespace

extern "C" {

LW_API int lw_attn_decode_noalloc(int fmt, const float* q, const void* K, const void* V, float* out,
                                  int64_t n_heads, int64_t n_kv_heads, int64_t head_dim, int64_t kv_len,
                                  float scale, void* stream) {
    if (fmt < LW_F16 || fmt > LW_MXFP4 || !lw::attn_fmt_supported(fmt)) return LW_EFMT;
    if (!q || !K || !V || !out) return LW_EINVAL;
    const int rc = lw::check_attn(fmt, n_heads, n_kv_heads, head_dim, kv_len, scale);
    if (rc != LW_OK) return rc;
    const lw::AttnPlan pl = lw::attn_plan(n_kv_heads, head_dim, kv_len, n_heads);
    if (pl.ws_bytes > kAttnScratchBytes) return LW_EINVAL;  // beyond the fixed scratch
    auto aligned = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; };
    if (!aligned(K, 256) || !aligned(V, 256) || !aligned(q, 16) || !aligned(out, 16)) return LW_EALIGN;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LW_EHIP;
    void* ws = scratch_ptr(dev);
    if (!ws) return LW_EHIP;
    const hipError_t err = lw::launch_attn(fmt, q, static_cast<const uint8_t*>(K), static_cast<const uint8_t*>(V), out,
                                           n_heads, n_kv_heads, head_dim, kv_len, scale, pl, static_cast<float*>(ws),
                                           reinterpret_cast<hipStream_t>(stream));
    return err == hipSuccess ? LW_OK : LW_EHIP;
}

}  // extern "C"
