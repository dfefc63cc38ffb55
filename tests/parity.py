"""Oracle references for the GPU parity tests: y and A, and the term mass F
of the form the selected kernel evaluates (gate.py derives the bound).

The VALU kernels evaluate the formats with an offset as s * sum q x +
mu * sum x (beta = 0); the matrix-core kernels multiply the bfloat16 of
128 + q (beta = 128). f16, Q8_0 and mxfp4 are plain sums of products (mxfp4
scaled by powers of two only): F is None. So is q1_0 on the matrix cores,
which multiply the exact bfloat16 +-1 of each bit and scale by d.
lw_kernel_name / lw_kernel_name_multi say which kernel a call launches."""
import numpy as np

from paper_2605_20706_amd import binding
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q8_0

MFMA_KERNELS = frozenset({"fewtok_kernel", "multitok_kernel", "multitok_pk_kernel", "skinny_kernel",
                          "gemm_kernel", "gemm32_kernel"})


def beta_of(kernel):
    return 128 if kernel.split("<")[0] in MFMA_KERNELS else 0


def plain(fmt):
    return fmt in (F16, Q8_0, MXFP4)


def plain_on(fmt, kernel):
    """The kernel's evaluation is a plain sum of products (no offset term)."""
    return plain(fmt) or (fmt == Q1_0 and beta_of(kernel) == 128)


def kernel_of(fmt, M, K, n_tok, Ms=None):
    """The kernel that computes the M-row matrix's outputs: the fused
    launch's kernel where lw_matvec_multi over Ms is one launch, else the
    kernel of the matrix's own lw_matvec."""
    if Ms is not None and len(Ms) > 1 and binding.launch_count_multi(fmt, list(Ms), K, n_tok) == 1:
        return binding.kernel_name_multi(fmt, list(Ms), K, n_tok)
    return binding.kernel_name(fmt, M, K, n_tok)


class Ref:
    """The oracle's y, A and both term masses (beta 0 and 128) of one matrix
    for a batch of tokens; F(kernel, nt) picks the one the kernel needs."""

    def __init__(self, oracle_mod, fmt, W, x, M, K, betas=(0, 128), n_threads=0):
        x = np.atleast_2d(x)
        self.fmt = fmt
        self.Fs = {}
        if plain(fmt):
            self.y, self.A, _ = oracle_mod.matvec(fmt, W, x, M, K, n_threads=n_threads)
            return
        for b in betas:
            y, A, F, _ = oracle_mod.matvec_f(fmt, W, x, M, K, b, n_threads=n_threads)
            self.y, self.A, self.Fs[b] = y, A, F

    def F(self, kernel, nt=None):
        if plain_on(self.fmt, kernel):
            return None
        F = self.Fs[beta_of(kernel)]
        return F if nt is None else F[:nt]


def reference(oracle_mod, fmt, W, x, M, K, kernel, n_threads=0):
    """(y, A, F) for one call whose first kernel is `kernel`."""
    r = Ref(oracle_mod, fmt, W, x, M, K, betas=(beta_of(kernel),), n_threads=n_threads)
    return r.y, r.A, r.F(kernel)


def block_max_mass(oracle_mod, fmt, W, x, M, K, rows=4096):
    """Bm[t][r] = sum_k |w_rk| * max over k's 32-block of |x_t| (float64),
    from the oracle's exact dequantization; the split term of the fp4 path's
    bound (tests/gate.py)."""
    x = np.atleast_2d(np.asarray(x, np.float64))
    xm = np.abs(x).reshape(x.shape[0], K // 32, 32).max(axis=2)  # [n_tok, K/32]
    Bm = np.empty((x.shape[0], M))
    Wd = oracle_mod.dequant(fmt, W, M * K).reshape(M, K)
    for r0 in range(0, M, rows):
        S = np.abs(Wd[r0:r0 + rows].astype(np.float64)).reshape(-1, K // 32, 32).sum(axis=2)  # [rows, K/32]
        Bm[:, r0:r0 + rows] = xm @ S.T
    return Bm
