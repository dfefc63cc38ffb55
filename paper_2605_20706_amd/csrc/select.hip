// Kernel selection table lookup and the sweep override (see select.hpp).
#include <cmath>
#include <cstdlib>

#include "lw.h"
#include "select.hpp"

namespace lw {
namespace {

struct SelEntry {
    int fmt;
    int n_tok;
    int64_t K, M;
    int cand;
};

#include "select_table.inc"

}  // namespace

int select_cand(int fmt, int64_t M, int64_t K, int64_t n_tok) {
    if (const char* f = std::getenv("LW_FORCE_CFG")) {
        const int v = std::atoi(f);
        if (v > 0) return v;
    }
    // Q4_1 shares Q4_0's code plane and kernels: it takes Q4_0's entries
    const int key = fmt == LW_Q4_1 ? LW_Q4_0 : fmt;
    int best = kCandDefault;
    double bd = 1.0 + 1e-9;  // |log2(M / entry M)| <= 1
    for (const SelEntry& e : kSelTable) {
        if (e.fmt != key || e.n_tok != n_tok || e.K != K) continue;
        const double d = std::fabs(std::log2((double)M / (double)e.M));
        if (d < bd) {
            bd = d;
            best = e.cand;
        }
    }
    return best;
}

}  // namespace lw
