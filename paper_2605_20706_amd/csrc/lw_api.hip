// C ABI of the lw library: argument validation and dispatch (see include/lw.h).
//
// Every check runs on the host before any HIP call, in the documented order
// (format, values, shape, alignment); a call that fails a check launches
// nothing. Dispatch: one or two tokens over the 4-bit formats with K a
// multiple of 2048 -> the VALU matrix-vector kernel with the activation in
// registers, where its table has an entry for the shape; else one token ->
// the VALU matrix-vector kernel with the activation in LDS; 2..16 tokens over
// the 4-bit formats -> the matrix-core kernel (token rows against 16 weight
// rows, one MFMA K step per 32-element block); Q8_0 with up to
// LW_GEMV_MAX_TOK tokens -> the VALU kernels, up to 16 -> the matrix-core
// kernel with K split across waves; more tokens -> the
// tiled matrix-core (prefill) kernel. The other quantized formats (Q5_0,
// Q5_1, Q5_K, Q6_K, Q2_K, MXFP4) run up to LW_GEMV_MAX_TOK tokens on the
// VALU kernels and more on the tiled matrix-core kernel. f16 and q1_0
// weights use the VALU kernel in token blocks for any token count.
// lw_matvec_ws (a workspace) sends LW_MXFP4 prefill to the fp4 matrix cores.
#include <cmath>

#include "lw_internal.hpp"
#include "select.hpp"

namespace {

bool known_fmt(int fmt) {
    return fmt >= LW_F16 && fmt <= LW_MXFP4;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// lw_matvec_multi takes the fused few-token launch from three tokens for the
// formats whose two-token calls run the register kernel (one launch per
// matrix is faster there at every shape), from two for the others.
bool fused_few(int fmt, int n_mat, int64_t n_tok) {
    const bool reg2 = fmt == LW_Q4_0 || fmt == LW_Q4_K || fmt == LW_Q4_1 || fmt == LW_Q1_0;
    return n_mat > 1 && n_tok <= 8 && n_tok >= (reg2 ? 3 : 2);
}

// The checks of lw_matvec that need no pointer, in the documented order.
int check_shape(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (M < 1 || K < 1 || n_tok < 1 || M > LW_MAX_DIM || K > LW_MAX_DIM || n_tok > LW_MAX_DIM) return LW_EINVAL;
    if (M > LW_MAX_ELEMS / K || n_tok > LW_MAX_ELEMS / K || n_tok > LW_MAX_ELEMS / M) return LW_EINVAL;
    if (K % 256) return LW_ESHAPE;
    return LW_OK;
}

// A matrix-core family candidate of the selection table (select.hpp), where
// it takes the call; hipErrorNotSupported otherwise (register-kernel
// candidates go through launch_gemv_reg, which reads the table itself).
hipError_t launch_family(int cand, int fmt, const uint8_t* Wb, const float* x, float* y, int64_t M, int64_t K,
                         int64_t n_tok, const lw::Planes& p, hipStream_t s) {
    const bool q4 = fmt == LW_Q4_0 || fmt == LW_Q4_K || fmt == LW_Q4_1;
    if (!q4) return hipErrorNotSupported;
    if (cand == lw::kCandFewtok && n_tok >= 2 && n_tok <= 8) return lw::launch_fewtok(fmt, Wb, x, y, M, K, n_tok, p, s);
    if (cand == lw::kCandMultitok && lw::multitok_supported(fmt, n_tok))
        return lw::launch_multitok(fmt, Wb, x, y, M, K, n_tok, p, s);
    if (cand == lw::kCandPrefill && n_tok >= 9) return lw::launch_prefill(fmt, Wb, x, y, M, K, n_tok, p, s);
    return hipErrorNotSupported;
}

// Kernel selection for a validated call: the swept table's candidate where
// it names one (select.hpp), else the built-in rules below.
// With a workspace (lw_matvec_ws), LW_MXFP4 prefill takes the fp4 matrix
// cores; every other call ignores it.
hipError_t dispatch(int fmt, const uint8_t* Wb, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                    hipStream_t s, uint8_t* ws = nullptr) {
    const lw::Planes p = lw::planes_of(fmt, M * K);
    if (ws && lw::fp4mm_takes(fmt, n_tok)) return lw::launch_fp4mm(Wb, x, y, M, K, n_tok, p, ws, s);
    hipError_t err = hipErrorNotSupported;
    const int cand = lw::select_cand(fmt, M, K, n_tok);
    if (cand >= lw::kCandFewtok) {
        err = launch_family(cand, fmt, Wb, x, y, M, K, n_tok, p, s);
        if (err != hipErrorNotSupported) return err;
    }
    if (n_tok <= 2) err = lw::launch_gemv_reg(fmt, Wb, x, y, M, K, n_tok, p, s);
    if (err == hipErrorNotSupported && n_tok >= 2 && n_tok <= 8) err = lw::launch_fewtok(fmt, Wb, x, y, M, K, n_tok, p, s);
    if (err == hipErrorNotSupported) {
        if (n_tok > 1 && lw::multitok_supported(fmt, n_tok))
            err = lw::launch_multitok(fmt, Wb, x, y, M, K, n_tok, p, s);
        else if (n_tok <= LW_GEMV_MAX_TOK)
            err = lw::launch_gemv(fmt, Wb, x, y, M, K, n_tok, p, s);
        else if (n_tok <= 16 && lw::skinny_supported(fmt))
            err = lw::launch_skinny(fmt, Wb, x, y, M, K, n_tok, p, s);
        else
            err = lw::launch_prefill(fmt, Wb, x, y, M, K, n_tok, p, s);
    }
    return err;
}

}  // namespace

namespace lw {

LaunchQuery& launch_query() {
    static thread_local LaunchQuery q;
    return q;
}

}  // namespace lw

extern "C" {

int64_t lw_weight_bytes(int fmt, int64_t n) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (n < 0 || n > LW_MAX_ELEMS) return LW_EINVAL;
    if (n % 256) return LW_ESHAPE;
    return lw::planes_of(fmt, n).total;
}

const char* lw_strerror(int code) {
    switch (code) {
    case LW_OK: return "success";
    case LW_EINVAL: return "invalid argument: null pointer or size out of range";
    case LW_EFMT: return "unknown weight format";
    case LW_ESHAPE: return "shape error: K (or n) must be a multiple of 256";
    case LW_EALIGN: return "alignment error: W must be 256-byte aligned, x/y/out 16-byte aligned";
    case LW_EHIP: return "HIP kernel launch failed";
    default: return "unknown error code";
    }
}

int lw_matvec(int fmt, const void* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
              void* stream) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (!W || !x || !y) return LW_EINVAL;
    const int rc = check_shape(fmt, M, K, n_tok);
    if (rc != LW_OK) return rc;
    if (!aligned(W, 256) || !aligned(x, 16) || !aligned(y, 16)) return LW_EALIGN;
    const hipError_t err = dispatch(fmt, static_cast<const uint8_t*>(W), x, y, M, K, n_tok,
                                    reinterpret_cast<hipStream_t>(stream));
    return err == hipSuccess ? LW_OK : LW_EHIP;
}

int64_t lw_matvec_workspace_bytes(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    const int rc = check_shape(fmt, M, K, n_tok);
    if (rc != LW_OK) return rc;
    return lw::fp4mm_takes(fmt, n_tok) ? lw::fp4mm_workspace_bytes(M, K, n_tok) : 0;
}

int lw_matvec_ws(int fmt, const void* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                 void* workspace, int64_t workspace_bytes, void* stream) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (!W || !x || !y) return LW_EINVAL;
    const int rc = check_shape(fmt, M, K, n_tok);
    if (rc != LW_OK) return rc;
    const int64_t need = lw::fp4mm_takes(fmt, n_tok) ? lw::fp4mm_workspace_bytes(M, K, n_tok) : 0;
    if (need > 0 && (!workspace || workspace_bytes < need)) return LW_EINVAL;
    if (!aligned(W, 256) || !aligned(x, 16) || !aligned(y, 16) || (need > 0 && !aligned(workspace, 256)))
        return LW_EALIGN;
    const hipError_t err = dispatch(fmt, static_cast<const uint8_t*>(W), x, y, M, K, n_tok,
                                    reinterpret_cast<hipStream_t>(stream),
                                    need > 0 ? static_cast<uint8_t*>(workspace) : nullptr);
    return err == hipSuccess ? LW_OK : LW_EHIP;
}

int lw_matvec_multi(int fmt, int n_mat, const void* const* W, float* const* y, const int64_t* M, const float* x,
                    int64_t K, int64_t n_tok, void* stream) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (!W || !y || !M || !x || n_mat < 1 || n_mat > LW_MULTI_MAX) return LW_EINVAL;
    for (int i = 0; i < n_mat; ++i)
        if (!W[i] || !y[i]) return LW_EINVAL;
    int worst = LW_OK;  // the first failing check in the documented order over all matrices
    for (int i = 0; i < n_mat; ++i) {
        const int rc = check_shape(fmt, M[i], K, n_tok);
        if (rc == LW_EINVAL) return LW_EINVAL;
        if (rc != LW_OK) worst = rc;
    }
    if (worst != LW_OK) return worst;
    if (!aligned(x, 16)) return LW_EALIGN;
    for (int i = 0; i < n_mat; ++i)
        if (!aligned(W[i], 256) || !aligned(y[i], 16)) return LW_EALIGN;
    const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t err = hipErrorNotSupported;
    const uint8_t* const* Wb = reinterpret_cast<const uint8_t* const*>(W);
    if (n_tok == 1 && n_mat > 1) err = lw::launch_gemv_multi(fmt, n_mat, Wb, y, M, x, K, s);
    if (fused_few(fmt, n_mat, n_tok)) err = lw::launch_fewtok_multi(fmt, n_mat, Wb, y, M, x, K, n_tok, s);
    if (err == hipErrorNotSupported) {
        err = hipSuccess;
        for (int i = 0; i < n_mat && err == hipSuccess; ++i)
            err = dispatch(fmt, static_cast<const uint8_t*>(W[i]), x, y[i], M[i], K, n_tok, s);
    }
    return err == hipSuccess ? LW_OK : LW_EHIP;
}

}  // extern "C"

namespace {

// Runs the selection of lw_matvec (n_mat == 0) or lw_matvec_multi with a
// launch query active: nothing is launched or dereferenced, the launchers
// stop at the launch. Returns false when the sizes fail the call's checks or
// the selection fails.
bool run_query(int fmt, int n_mat, const int64_t* Ms, int64_t M, int64_t K, int64_t n_tok, lw::LaunchQuery& out,
               bool with_ws = false) {
    if (n_mat == 0) {
        if (check_shape(fmt, M, K, n_tok) != LW_OK) return false;
    } else {
        if (!Ms || n_mat < 1 || n_mat > LW_MULTI_MAX) return false;
        for (int i = 0; i < n_mat; ++i)
            if (check_shape(fmt, Ms[i], K, n_tok) != LW_OK) return false;
    }
    lw::LaunchQuery& q = lw::launch_query();
    q.active = true;
    q.name = nullptr;
    q.count = 0;
    alignas(256) static const uint8_t stand_in[256] = {};
    const float* xs = reinterpret_cast<const float*>(stand_in);
    float* ys0 = const_cast<float*>(xs);
    hipError_t err;
    if (n_mat == 0) {
        err = dispatch(fmt, stand_in, xs, ys0, M, K, n_tok, nullptr,
                       with_ws ? const_cast<uint8_t*>(stand_in) : nullptr);
    } else {
        // the same routing as lw_matvec_multi
        const uint8_t* Ws[LW_MULTI_MAX];
        float* ys[LW_MULTI_MAX];
        for (int i = 0; i < LW_MULTI_MAX; ++i) {
            Ws[i] = stand_in;
            ys[i] = ys0;
        }
        err = hipErrorNotSupported;
        if (n_tok == 1 && n_mat > 1) err = lw::launch_gemv_multi(fmt, n_mat, Ws, ys, Ms, xs, K, nullptr);
        if (fused_few(fmt, n_mat, n_tok)) err = lw::launch_fewtok_multi(fmt, n_mat, Ws, ys, Ms, xs, K, n_tok, nullptr);
        if (err == hipErrorNotSupported) {
            err = hipSuccess;
            for (int i = 0; i < n_mat && err == hipSuccess; ++i)
                err = dispatch(fmt, stand_in, xs, ys0, Ms[i], K, n_tok, nullptr);
        }
    }
    out = q;
    q.active = false;
    return err == hipSuccess;
}

}  // namespace

extern "C" {

const char* lw_kernel_name(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    lw::LaunchQuery r;
    return run_query(fmt, 0, nullptr, M, K, n_tok, r) ? r.name : nullptr;
}

const char* lw_kernel_name_multi(int fmt, int n_mat, const int64_t* M, int64_t K, int64_t n_tok) {
    lw::LaunchQuery r;
    return run_query(fmt, n_mat, M, 0, K, n_tok, r) ? r.name : nullptr;
}

int64_t lw_launch_count(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    const int rc = check_shape(fmt, M, K, n_tok);
    if (rc != LW_OK) return rc;
    lw::LaunchQuery r;
    return run_query(fmt, 0, nullptr, M, K, n_tok, r) ? r.count : LW_EHIP;
}

const char* lw_kernel_name_ws(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    lw::LaunchQuery r;
    return run_query(fmt, 0, nullptr, M, K, n_tok, r, true) ? r.name : nullptr;
}

int64_t lw_launch_count_ws(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    const int rc = check_shape(fmt, M, K, n_tok);
    if (rc != LW_OK) return rc;
    lw::LaunchQuery r;
    return run_query(fmt, 0, nullptr, M, K, n_tok, r, true) ? r.count : LW_EHIP;
}

int64_t lw_launch_count_multi(int fmt, int n_mat, const int64_t* M, int64_t K, int64_t n_tok) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (!M || n_mat < 1 || n_mat > LW_MULTI_MAX) return LW_EINVAL;
    int worst = LW_OK;
    for (int i = 0; i < n_mat; ++i) {
        const int rc = check_shape(fmt, M[i], K, n_tok);
        if (rc == LW_EINVAL) return LW_EINVAL;
        if (rc != LW_OK) worst = rc;
    }
    if (worst != LW_OK) return worst;
    lw::LaunchQuery r;
    return run_query(fmt, n_mat, M, 0, K, n_tok, r) ? r.count : LW_EHIP;
}

}  // extern "C"

namespace {

}  // namespace

namespace lw {

// The checks of lw_attn_decode that need no pointer, in the documented order.
int check_attn(int fmt, int64_t n_heads, int64_t n_kv, int64_t head_dim, int64_t kv_len, float scale) {
    if (fmt < LW_F16 || fmt > LW_MXFP4 || !lw::attn_fmt_supported(fmt)) return LW_EFMT;
    if (n_heads < 1 || n_kv < 1 || kv_len < 1 || n_heads > 4096 || kv_len >= ((int64_t)1 << 31) ||
        n_kv * kv_len > LW_MAX_ELEMS / 128)
        return LW_EINVAL;
    if (n_heads % n_kv) return LW_EINVAL;
    const int64_t grp = n_heads / n_kv;
    if (grp != 1 && grp != 2 && grp != 4 && grp != 8) return LW_EINVAL;
    if (head_dim != 64 && head_dim != 128) return LW_EINVAL;
    if (!std::isfinite(scale)) return LW_EINVAL;
    if ((n_kv * kv_len * head_dim) % 256) return LW_ESHAPE;
    return LW_OK;
}

}  // namespace lw

extern "C" {

int64_t lw_attn_workspace_bytes(int fmt, int64_t n_heads, int64_t n_kv_heads, int64_t head_dim, int64_t kv_len) {
    const int rc = lw::check_attn(fmt, n_heads, n_kv_heads, head_dim, kv_len, 1.0f);
    if (rc != LW_OK) return rc;
    return lw::attn_plan(n_kv_heads, head_dim, kv_len, n_heads).ws_bytes;
}

const char* lw_attn_kernel_name(int fmt, int64_t n_heads, int64_t n_kv_heads, int64_t head_dim, int64_t kv_len) {
    if (lw::check_attn(fmt, n_heads, n_kv_heads, head_dim, kv_len, 1.0f) != LW_OK) return nullptr;
    const lw::AttnPlan pl = lw::attn_plan(n_kv_heads, head_dim, kv_len, n_heads);
    lw::LaunchQuery& q = lw::launch_query();
    q.active = true;
    q.name = nullptr;
    q.count = 0;
    alignas(256) static const uint8_t stand_in[256] = {};
    float* fs = reinterpret_cast<float*>(const_cast<uint8_t*>(stand_in));
    const hipError_t err = lw::launch_attn(fmt, fs, stand_in, stand_in, fs, n_heads, n_kv_heads, head_dim, kv_len,
                                           1.0f, pl, fs, nullptr);
    const char* name = q.name;
    q.active = false;
    return err == hipSuccess ? name : nullptr;
}

int lw_attn_decode(int fmt, const float* q, const void* K, const void* V, float* out, int64_t n_heads,
                   int64_t n_kv_heads, int64_t head_dim, int64_t kv_len, float scale, void* workspace,
                   int64_t workspace_bytes, void* stream) {
    if (!known_fmt(fmt) || !lw::attn_fmt_supported(fmt)) return LW_EFMT;
    if (!q || !K || !V || !out || !workspace) return LW_EINVAL;
    const int rc = lw::check_attn(fmt, n_heads, n_kv_heads, head_dim, kv_len, scale);
    if (rc != LW_OK) return rc;
    const lw::AttnPlan pl = lw::attn_plan(n_kv_heads, head_dim, kv_len, n_heads);
    if (workspace_bytes < pl.ws_bytes) return LW_EINVAL;
    if (!aligned(K, 256) || !aligned(V, 256) || !aligned(q, 16) || !aligned(out, 16) || !aligned(workspace, 16))
        return LW_EALIGN;
    const hipError_t err = lw::launch_attn(fmt, q, static_cast<const uint8_t*>(K), static_cast<const uint8_t*>(V), out,
                                           n_heads, n_kv_heads, head_dim, kv_len, scale, pl,
                                           static_cast<float*>(workspace), reinterpret_cast<hipStream_t>(stream));
    return err == hipSuccess ? LW_OK : LW_EHIP;
}

int lw_dequant(int fmt, const void* W, float* out, int64_t n) {
    if (!known_fmt(fmt)) return LW_EFMT;
    if (!W || !out) return LW_EINVAL;
    if (n < 0 || n > LW_MAX_ELEMS) return LW_EINVAL;
    if (n % 256) return LW_ESHAPE;
    if (!aligned(W, 256) || !aligned(out, 16)) return LW_EALIGN;
    if (n == 0) return LW_OK;
    const lw::Planes p = lw::planes_of(fmt, n);
    const hipError_t err = lw::launch_dequant(fmt, static_cast<const uint8_t*>(W), out, n, p, nullptr);
    return err == hipSuccess ? LW_OK : LW_EHIP;
}

}  // extern "C"
