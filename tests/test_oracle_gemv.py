"""Pins of the oracle's matrix-vector product (Sec. 2.1: decode computes
y = W . x for the dequantized W).

Checked against numpy's float64 matmul of the oracle's own (separately
pinned) dequantized matrix, and against properties the definition fixes: a
one-hot x returns a column of W bit-exactly, x of ones returns row sums,
linearity in x, exact scaling by powers of two, thread-count invariance and
agreement of the sampled and full forms.
"""
import numpy as np
import pytest

from paper_2605_20706_amd import layout, synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

ALL = [F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4]


def make(fmt, M, K, seed):
    rng = np.random.default_rng(seed)
    f = synth.gen_fields(fmt, M * K, rng)
    return synth.pack_fields(fmt, f), f


@pytest.mark.parametrize("fmt", ALL)
@pytest.mark.parametrize("M,K,n_tok", [(1, 256, 1), (7, 512, 3), (33, 256, 2), (5, 768, 1)])
def test_brute_force_vs_numpy(oracle_mod, fmt, M, K, n_tok):
    W, _ = make(fmt, M, K, 100 + M + K + fmt)
    x = synth.gen_x_seeded(5 + M, K, n_tok)
    y, A, _ = oracle_mod.matvec(fmt, W, x, M, K)
    Wd = oracle_mod.dequant(fmt, W, M * K).reshape(M, K).astype(np.float64)
    ref = x.astype(np.float64) @ Wd.T                  # [n_tok, M]
    refA = np.abs(x.astype(np.float64)) @ np.abs(Wd).T
    assert y.shape == (n_tok, M)
    assert np.allclose(y, ref, rtol=0, atol=1e-12 * refA.max())
    assert np.allclose(A, refA, rtol=1e-12, atol=0)


@pytest.mark.parametrize("fmt", ALL)
def test_one_hot_returns_column_bit_exact(oracle_mod, fmt):
    M, K = 9, 512
    W, _ = make(fmt, M, K, 21)
    Wd = oracle_mod.dequant(fmt, W, M * K).reshape(M, K)
    for k in (0, 17, 255, 256, 511):
        x = np.zeros((1, K), np.float32)
        x[0, k] = 1.0
        y, _, _ = oracle_mod.matvec(fmt, W, x, M, K)
        assert np.array_equal(y[0], Wd[:, k].astype(np.float64))


@pytest.mark.parametrize("fmt", ALL)
def test_ones_gives_row_sums(oracle_mod, fmt):
    M, K = 6, 1024
    W, _ = make(fmt, M, K, 22)
    Wd = oracle_mod.dequant(fmt, W, M * K).reshape(M, K).astype(np.float64)
    y, A, _ = oracle_mod.matvec(fmt, W, np.ones((1, K), np.float32), M, K)
    assert np.allclose(y[0], Wd.sum(axis=1), rtol=0, atol=1e-13 * np.abs(Wd).sum(axis=1).max())
    assert np.allclose(A[0], np.abs(Wd).sum(axis=1), rtol=1e-14)


@pytest.mark.parametrize("fmt", ALL)
def test_linearity_and_token_independence(oracle_mod, fmt):
    M, K = 11, 512
    W, _ = make(fmt, M, K, 23)
    a = synth.gen_x_seeded(1, K)
    b = synth.gen_x_seeded(2, K)
    ya, Aa, _ = oracle_mod.matvec(fmt, W, a, M, K)
    yb, Ab, _ = oracle_mod.matvec(fmt, W, b, M, K)
    yab, _, _ = oracle_mod.matvec(fmt, W, np.concatenate([a, b]), M, K)
    assert np.array_equal(yab[0], ya[0]) and np.array_equal(yab[1], yb[0])
    # 2a + b is exact in float32 for these magnitudes only up to rounding: use the A bound
    c = (np.float32(2) * a + b)
    yc, _, _ = oracle_mod.matvec(fmt, W, c, M, K)
    assert np.allclose(yc[0], 2 * ya[0] + yb[0], rtol=0, atol=1e-6 * (2 * Aa[0] + Ab[0]).max())


@pytest.mark.parametrize("fmt", [Q8_0, Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4])
def test_power_of_two_scale(oracle_mod, fmt):
    """Doubling every binary16 scale and min (exponent + 1, no overflow)
    doubles y exactly."""
    M, K = 8, 512
    rng = np.random.default_rng(24)
    f = synth.gen_fields(fmt, M * K, rng)
    W = synth.pack_fields(fmt, f)
    f2 = dict(f)
    for key in (("d", "m") if fmt in (Q4_1, Q5_1) else ("d", "dmin")):
        if key in f2:
            f2[key] = (f2[key].astype(np.float64) * 2).astype(np.float16)
    if fmt == MXFP4:
        f2["E"] = (f2["E"] + 1).astype(np.uint8)  # e8m0 exponent + 1: the block scale doubles
    W2 = synth.pack_fields(fmt, f2)
    x = synth.gen_x_seeded(9, K, 2)
    y, _, _ = oracle_mod.matvec(fmt, W, x, M, K)
    y2, _, _ = oracle_mod.matvec(fmt, W2, x, M, K)
    assert np.array_equal(y2, 2 * y)


def test_threads_and_sampled_agree(oracle_mod):
    M, K, n_tok = 37, 1024, 3
    W, _ = make(Q4_K, M, K, 25)
    x = synth.gen_x_seeded(10, K, n_tok)
    y1, A1, T1 = oracle_mod.matvec(Q4_K, W, x, M, K, n_threads=1)
    y8, A8, T8 = oracle_mod.matvec(Q4_K, W, x, M, K, n_threads=8)
    assert T1 == 1 and T8 == 8
    assert np.array_equal(y1, y8) and np.array_equal(A1, A8)
    rows = np.array([0, 36, 5, 17])
    toks = np.array([2, 0, 1, 2])
    ys, As = oracle_mod.matvec_sampled(Q4_K, W, x, M, K, rows, toks)
    assert np.array_equal(ys, y1[toks, rows]) and np.array_equal(As, A1[toks, rows])


def test_rejects_bad_arguments(oracle_mod):
    W, _ = make(Q4_0, 4, 256, 26)
    with pytest.raises(ValueError):
        oracle_mod.matvec(Q4_0, W, np.zeros((1, 255), np.float32), 4, 255)
    with pytest.raises(ValueError):
        oracle_mod.dequant(9, W, 256)
    with pytest.raises(ValueError):
        oracle_mod.matvec_sampled(Q4_0, W, np.zeros((1, 256), np.float32), 4, 256, [4], [0])
