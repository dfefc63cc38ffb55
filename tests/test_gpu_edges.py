"""The method's edge cases on every kernel family, against the oracle.

Inputs the uniform synthetic draws never produce:
  * rows whose dequantized weights are all exactly zero while their scales
    are not (q4_0 codes 8; q4_1 codes 4 with m = -4d; q4_k codes 3 with
    dmin = d and m_j = 3 sc_j; q8_0 codes 0; f16 zeros; q1_0, which has no
    zero level, with d = 0): A = 0 there, and a factored evaluation returns a
    rounding residue bounded by 2^-17 * F (tests/gate.py), not exactly 0;
  * blocks whose scale is 0 (d = 0; for q4_k also d = dmin = 0);
  * weights drawn from N(0, 0.02^2) and encoded by an Eq. (1) quantizer, so
    the codes peak at the code of zero (the factored forms' worst case for
    the error relative to A);
  * activations scaled by 2^60 and 2^-60 (every product and partial sum stays
    in float32's normal range there, so the bound holds unchanged).

Each case names the kernel family it exercises (lw_kernel_name); the CPU test
in test_abi.py checks that the table covers every family."""
import numpy as np
import pytest

import gate
from gpu_util import gpu_dequant, same_bits_or_both_zero, to_gpu
from parity import Ref, kernel_of
from paper_2605_20706_amd import binding, synth

pytestmark = pytest.mark.gpu

FMTS = [0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11]
# (M, K, n_tok): the single-token LDS kernel; the register kernel (one chunk,
# two tokens, seven chunks over seven waves); the pair-step and few-token
# matrix-core kernels; the 9..16-token kernels (multitok, Q8_0 skinny, VALU
# token blocks); prefill (gemm32 with a K split, Q8_0 gemm, token blocks).
EDGE_SHAPES = [(300, 2304, 1), (3000, 2048, 1), (2000, 2048, 2), (4100, 14336, 1), (300, 2304, 5),
               (8200, 4096, 4), (300, 2304, 12), (1100, 4352, 40)]
# lw_matvec_multi: the fused single-token launch and the fused few-token launch.
EDGE_MULTI = [((3000, 2000), 2048, 1), ((8200, 8200), 4096, 4)]
KINDS = ["zero_rows", "zero_scales", "eq1_normal", "x_times_2^60", "x_times_2^-60"]


def fields_for(kind, fmt, M, K, seed):
    rng = np.random.default_rng([seed, fmt, M, K, KINDS.index(kind)])
    n = M * K
    if kind == "zero_rows":
        f = synth.gen_fields_eq1(fmt, n, rng)
        rows = np.unique(np.concatenate([[0, 1, M // 2, M - 1], rng.integers(0, M, max(1, M // 64))]))
        return synth.zero_rows(fmt, f, rows, K), rows
    if kind == "zero_scales":
        return synth.zero_scales(fmt, synth.gen_fields(fmt, n, rng), rng), None
    if kind == "eq1_normal":
        return synth.gen_fields_eq1(fmt, n, rng), None
    return synth.gen_fields(fmt, n, rng), None


def x_for(kind, K, n_tok, seed):
    x = synth.gen_x_seeded([seed, K, n_tok, 77], K, n_tok)
    if kind == "x_times_2^60":
        x = (x.astype(np.float64) * 2.0 ** 60).astype(np.float32)
    elif kind == "x_times_2^-60":
        x = (x.astype(np.float64) * 2.0 ** -60).astype(np.float32)
    return x


def check_kind(oracle_mod, kind, fmt, y, W, x, M, K, kern, zrows, what):
    ref = Ref(oracle_mod, fmt, W, x, M, K)
    m = gate.check(y, ref.y, ref.A, ref.F(kern), f32_bound=1e-4, what=what)
    if zrows is not None:
        assert (ref.A[:, zrows] == 0).all(), what
        zr = np.abs(np.asarray(y, np.float64)[:, zrows])
        F = ref.F(kern)
        if F is None:
            assert (zr == 0).all(), (what, "a plain sum of zeros must be exactly 0")
        else:
            assert (zr <= gate.C_FACTORED * F[:, zrows]).all(), (what, float(zr.max()))
    print("  %-14s %s scaled=%.3g f32_ratio=%.3g zero_rows=%d" % (kind, kern, m["scaled"], m["f32_ratio"],
                                                                  m["zero_rows"]), flush=True)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,K,n_tok", EDGE_SHAPES)
def test_edge_inputs(oracle_mod, fmt, M, K, n_tok):
    import torch
    kern = kernel_of(fmt, M, K, n_tok)
    print("edges fmt=%d M=%d K=%d n_tok=%d kernel=%s" % (fmt, M, K, n_tok, kern), flush=True)
    for kind in KINDS:
        f, zrows = fields_for(kind, fmt, M, K, 81)
        W = synth.pack_fields(fmt, f)
        x = x_for(kind, K, n_tok, 82)
        y = binding.matvec(fmt, to_gpu(W), to_gpu(x), M, K)
        torch.cuda.synchronize()
        check_kind(oracle_mod, kind, fmt, y.cpu().numpy(), W, x, M, K, kern, zrows, (kind, fmt, M, K, n_tok, kern))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("Ms,K,n_tok", EDGE_MULTI)
def test_edge_inputs_multi(oracle_mod, fmt, Ms, K, n_tok):
    import torch
    kern = kernel_of(fmt, Ms[0], K, n_tok, Ms=Ms)
    print("edges multi fmt=%d Ms=%s K=%d n_tok=%d kernel=%s" % (fmt, Ms, K, n_tok, kern), flush=True)
    for kind in ("zero_rows", "eq1_normal", "x_times_2^-60"):
        fs = [fields_for(kind, fmt, m, K, 90 + i) for i, m in enumerate(Ms)]
        Ws = [synth.pack_fields(fmt, f) for f, _ in fs]
        x = x_for(kind, K, n_tok, 91)
        ys = binding.matvec_multi(fmt, [to_gpu(w) for w in Ws], to_gpu(x), list(Ms), K)
        torch.cuda.synchronize()
        for i, m in enumerate(Ms):
            check_kind(oracle_mod, kind, fmt, ys[i].cpu().numpy(), Ws[i], x, m, K, kern, fs[i][1],
                       (kind, fmt, Ms, K, n_tok, i, kern))


@pytest.mark.parametrize("fmt", FMTS)
def test_edge_dequant_bit_exact(oracle_mod, fmt):
    """lw_dequant on zero rows, zero scales and Eq. (1)-encoded weights: bit
    for bit the oracle's values (+0 = -0)."""
    M, K = 96, 2304
    for kind in ("zero_rows", "zero_scales", "eq1_normal"):
        f, _ = fields_for(kind, fmt, M, K, 95)
        W = synth.pack_fields(fmt, f)
        got = gpu_dequant(fmt, W, M * K)
        ref = oracle_mod.dequant(fmt, W, M * K)
        assert same_bits_or_both_zero(got, ref).all(), (kind, fmt)
