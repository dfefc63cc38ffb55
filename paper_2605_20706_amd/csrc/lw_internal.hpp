// Host-side declarations shared by the C-ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "lw.h"

namespace lw {

// Kernel-name query (lw_kernel_name, lw_launch_count). While a query is
// active on the calling thread the launchers launch nothing: at the point
// where they would launch, they record the kernel's name (the first one, when
// a call launches several), add the launches they would make to the count and
// return hipSuccess. So a query walks exactly the selection a real call
// makes.
struct LaunchQuery {
    bool active = false;
    const char* name = nullptr;
    int64_t count = 0;
};
LaunchQuery& launch_query();

// True when a query is active (the caller returns hipSuccess instead of
// launching); records name if none is recorded yet and counts `launches`
// kernel launches (a launcher that would also launch a fill kernel passes 2).
inline bool query_only(const char* name, int launches = 1) {
    LaunchQuery& q = launch_query();
    if (!q.active) return false;
    if (!q.name) q.name = name;
    q.count += launches;
    return true;
}

// "base<V0, V1, ...>": the template part of a kernel's demangled name, built
// once per instantiation (Tag::base names the kernel template).
template <class Tag, int... V>
const char* kernel_name() {
    static const std::string s = [] {
        std::string r = std::string(Tag::base) + "<";
        const int v[] = {V...};
        for (size_t i = 0; i < sizeof...(V); ++i) r += (i ? ", " : "") + std::to_string(v[i]);
        return r + ">";
    }();
    return s.c_str();
}

// Byte offsets of planes 1, 2 and 3 and the total size of n packed elements of
// fmt (split-plane layout: later planes start at the end of the previous one
// rounded up to 256 bytes). n must already be valid for fmt.
struct Planes {
    int64_t off1 = 0, off2 = 0, off3 = 0, total = 0;
};

inline int64_t round_up_256(int64_t v) { return (v + 255) / 256 * 256; }

inline Planes planes_of(int fmt, int64_t n) {
    Planes p;
    switch (fmt) {
    case LW_F16:
        p.total = 2 * n;
        break;
    case LW_Q8_0:
        p.off1 = round_up_256(n);
        p.total = p.off1 + 2 * (n / 32);
        break;
    case LW_Q4_0:
        p.off1 = round_up_256(n / 2);
        p.total = p.off1 + 2 * (n / 32);
        break;
    case LW_Q4_1:
        p.off1 = round_up_256(n / 2);
        p.total = p.off1 + 4 * (n / 32);
        break;
    case LW_Q1_0:
        p.off1 = round_up_256(n / 8);
        p.total = p.off1 + 2 * (n / 128);
        break;
    case LW_Q4_K:
        p.off1 = round_up_256(n / 2);
        p.off2 = round_up_256(p.off1 + 12 * (n / 256));
        p.total = p.off2 + 4 * (n / 256);
        break;
    case LW_Q5_0:
    case LW_Q5_1:
        p.off1 = round_up_256(n / 2);
        p.off2 = round_up_256(p.off1 + n / 8);
        p.total = p.off2 + (fmt == LW_Q5_0 ? 2 : 4) * (n / 32);
        break;
    case LW_Q5_K:
        p.off1 = round_up_256(n / 2);
        p.off2 = round_up_256(p.off1 + n / 8);
        p.off3 = round_up_256(p.off2 + 12 * (n / 256));
        p.total = p.off3 + 4 * (n / 256);
        break;
    case LW_Q6_K:
        p.off1 = round_up_256(n / 2);
        p.off2 = round_up_256(p.off1 + n / 4);
        p.off3 = round_up_256(p.off2 + n / 16);
        p.total = p.off3 + 2 * (n / 256);
        break;
    case LW_MXFP4:
        p.off1 = round_up_256(n / 2);
        p.total = p.off1 + n / 32;
        break;
    case LW_Q2_K:
        p.off1 = round_up_256(n / 4);
        p.off2 = round_up_256(p.off1 + n / 16);
        p.total = p.off2 + 4 * (n / 256);
        break;
    default:
        break;
    }
    return p;
}

// Rows of up to kMaxSegs matrices that share the same activations, seen by a
// kernel as one row space (lw_matvec_multi): segment i holds the global rows
// [start[i], start[i] + M[i]) of weights W[i] (plane offsets off1[i],
// off2[i]) and writes y[i]. Unused segments start past every row. Kernels
// that give each workgroup rows of one matrix only use wg0[i], the first
// workgroup of segment i, instead of start.
constexpr int kMaxSegs = LW_MULTI_MAX;
template <int NS>
struct RowSegs {
    const uint8_t* W[NS];
    float* y[NS];
    int64_t off1[NS], off2[NS], off3[NS], start[NS], M[NS], wg0[NS];
};

// Kernel launchers. Arguments are already validated; each returns the
// hipError_t of its launch.
hipError_t launch_dequant(int fmt, const uint8_t* W, float* out, int64_t n, const Planes& p,
                          hipStream_t stream);
hipError_t launch_gemv(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                       int64_t n_tok, const Planes& p, hipStream_t stream);
// Any n_tok >= 1 on the matrix-vector kernels: whole token blocks in one
// launch (grid.y = block), the remaining tokens in one more.
hipError_t launch_gemv_blocks(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                              int64_t n_tok, const Planes& p, hipStream_t stream);
// One launch of a single-token kernel over the rows of n matrices that share
// x (one token, same format and K); hipErrorNotSupported when the shapes are
// not ones the single-token kernels take as one row space.
hipError_t launch_gemv_multi(int fmt, int n, const uint8_t* const* W, float* const* y, const int64_t* M,
                             const float* x, int64_t K, hipStream_t stream);
// Register-resident-activation kernel (4-bit formats, one or two tokens, K a
// multiple of 2048 with a table entry); hipErrorNotSupported when the shape
// is not one it takes.
hipError_t launch_gemv_reg(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                           int64_t n_tok, const Planes& p, hipStream_t stream);
// Matrix-core path for 2 <= n_tok <= 16 with streamed weights (4-bit and 8-bit formats).
bool skinny_supported(int fmt);
hipError_t launch_skinny(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                         int64_t n_tok, const Planes& p, hipStream_t stream);
// Matrix-core path for 2 <= n_tok <= 16 over the 4-bit formats (token rows
// against 16 weight rows per MFMA; weights streamed once).
bool multitok_supported(int fmt, int64_t n_tok);
hipError_t launch_multitok(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                           int64_t n_tok, const Planes& p, hipStream_t stream);
// Matrix-core path for 2 <= n_tok <= 8 over the 4-bit formats with the
// activations converted once per workgroup into LDS; hipErrorNotSupported
// when the call is not one it takes.
hipError_t launch_fewtok(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                         int64_t n_tok, const Planes& p, hipStream_t stream);
// The same over the rows of n matrices that share x (lw_matvec_multi).
hipError_t launch_fewtok_multi(int fmt, int n, const uint8_t* const* W, float* const* y, const int64_t* M,
                               const float* x, int64_t K, int64_t n_tok, hipStream_t stream);
// Decode attention over a KV cache in a weight format (attn.hip): the split
// of the kv_len positions over workgroups (rps positions per split) and the
// workspace it needs, the formats it takes, and the two launches.
struct AttnPlan {
    int64_t splits = 0, rps = 0, ws_bytes = 0;
};
AttnPlan attn_plan(int64_t n_kv, int64_t head_dim, int64_t kv_len, int64_t n_heads);
bool attn_fmt_supported(int fmt);
// lw_attn_decode's checks that need no pointer, in the documented order
// (LW_EFMT, LW_EINVAL, LW_ESHAPE); LW_OK when they pass.
int check_attn(int fmt, int64_t n_heads, int64_t n_kv, int64_t head_dim, int64_t kv_len, float scale);
hipError_t launch_attn(int fmt, const float* q, const uint8_t* K, const uint8_t* V, float* out, int64_t n_heads,
                       int64_t n_kv, int64_t head_dim, int64_t kv_len, float scale, const AttnPlan& pl, float* ws,
                       hipStream_t stream);
// Work split of a tiled matrix-core launch: nrt x ntt (row tile, token tile)
// pairs, ks K splits of sbp super-blocks each (the last one possibly
// shorter); plan_split picks the fewest splits that keep the compute units
// busy (prefill.hip). A K-split launch adds its partial results atomically
// into y, which zero_fill clears first.
struct GemmSplit {
    int64_t nrt, ntt;
    int ks, sbp;
};
GemmSplit plan_split(int64_t nrt, int64_t ntt, int64_t K, int64_t cus = 0);  // cus 0: the device's
void zero_fill(float* y, int64_t n, hipStream_t stream);
// Matrix-core path for larger token counts (prefill).
hipError_t launch_prefill(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                          int64_t n_tok, const Planes& p, hipStream_t stream);
// LW_MXFP4 prefill on the fp4 x fp6 matrix cores (fp4mm.hip): the activations
// are first split into e2m3 pieces in a caller-provided workspace of
// fp4mm_workspace_bytes; fp4mm_takes says whether a call runs there.
bool fp4mm_takes(int fmt, int64_t n_tok);
int64_t fp4mm_workspace_bytes(int64_t M, int64_t K, int64_t n_tok);
hipError_t launch_fp4mm(const uint8_t* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                        const Planes& p, uint8_t* ws, hipStream_t stream);

}  // namespace lw
