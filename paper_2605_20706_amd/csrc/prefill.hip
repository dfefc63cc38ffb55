// Multi-token path for n_tok > LW_GEMV_MAX_TOK: token blocks of the
// matrix-vector kernel (placeholder until the matrix-core kernel lands).
#include "lw_internal.hpp"

namespace lw {

hipError_t launch_prefill(int fmt, const uint8_t* W, const float* x, float* y, int64_t M, int64_t K,
                          int64_t n_tok, const Planes& p, hipStream_t stream) {
    for (int64_t t0 = 0; t0 < n_tok; t0 += LW_GEMV_MAX_TOK) {
        const int64_t nt = (n_tok - t0) < LW_GEMV_MAX_TOK ? (n_tok - t0) : LW_GEMV_MAX_TOK;
        const hipError_t err = launch_gemv(fmt, W, x + t0 * K, y + t0 * M, M, K, nt, p, stream);
        if (err != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace lw
