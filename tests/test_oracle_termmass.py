"""Pins of the oracle's term mass F (the scale of a factored evaluation's
rounding error, tests/gate.py).

F = sum_k (|s_k| (q_k + beta) + |mu_k - beta s_k|) |x_k| for Eq. (1)'s scale
s and offset mu of each element and its stored unsigned code q. Every pin
ties F to the condition sum A = sum |w x| of other matrices (A itself is
pinned against numpy's float64 product in test_oracle_gemv.py) or to a
property the definition fixes: F = A for the formats without an offset,
F >= A (triangle inequality), and F growing linearly in beta by 2 * sum |s x|
when s and -mu are non-negative."""
import numpy as np
import pytest

from paper_2605_20706_amd import synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

M, K = 9, 512


def fields(fmt, seed):
    return synth.gen_fields(fmt, M * K, np.random.default_rng([seed, fmt]))


def A_of(oracle_mod, fmt, f, x):
    _, A, _ = oracle_mod.matvec(fmt, synth.pack_fields(fmt, f), x, M, K)
    return A


def F_of(oracle_mod, fmt, f, x, beta):
    _, _, F, _ = oracle_mod.matvec_f(fmt, synth.pack_fields(fmt, f), x, M, K, beta)
    return F


@pytest.mark.parametrize("fmt", [F16, Q8_0, MXFP4])
@pytest.mark.parametrize("beta", [0, 128])
def test_no_offset_formats_have_F_equal_A(oracle_mod, fmt, beta):
    f = fields(fmt, 1)
    x = synth.gen_x_seeded(2, K, 3)
    assert np.array_equal(F_of(oracle_mod, fmt, f, x, beta), A_of(oracle_mod, fmt, f, x))


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K])
@pytest.mark.parametrize("beta", [0, 1, 128])
def test_F_at_least_A(oracle_mod, fmt, beta):
    f = fields(fmt, 3)
    x = synth.gen_x_seeded(4, K, 2)
    F = F_of(oracle_mod, fmt, f, x, beta)
    A = A_of(oracle_mod, fmt, f, x)
    assert (F >= A * (1 - 1e-12)).all()


def test_q4_1_without_min_has_F_equal_A(oracle_mod):
    f = fields(Q4_1, 5)
    f["m"][:] = np.float16(0)
    x = synth.gen_x_seeded(6, K, 2)
    assert np.allclose(F_of(oracle_mod, Q4_1, f, x, 0), A_of(oracle_mod, Q4_1, f, x), rtol=1e-13, atol=0)


def test_q4_0_against_condition_sums(oracle_mod):
    """F_beta = sum |d| (q + 8 + 2 beta) |x| = A(d, codes q, as q4_1 with m = 0)
    + (8 + 2 beta) * A(d, all codes 9, i.e. values d)."""
    f = fields(Q4_0, 7)
    x = synth.gen_x_seeded(8, K, 3)
    a_q = A_of(oracle_mod, Q4_1, {"q": f["q"], "d": f["d"], "m": np.zeros_like(f["d"])}, x)
    a_1 = A_of(oracle_mod, Q4_0, {"q": np.full_like(f["q"], 9), "d": f["d"]}, x)
    for beta in (0, 3, 128):
        F = F_of(oracle_mod, Q4_0, f, x, beta)
        assert np.allclose(F, a_q + (8 + 2 * beta) * a_1, rtol=1e-12, atol=0), beta


def test_q4_1_against_condition_sums(oracle_mod):
    """Mins m <= 0 (the recipe's range): F_beta = sum (d (q + beta) + |m| + beta d) |x|
    = A(codes q, m = 0) + A(codes 0: values m) + 2 beta A(codes 1, m = 0)."""
    f = fields(Q4_1, 9)
    assert (f["m"].astype(np.float64) <= 0).all()
    x = synth.gen_x_seeded(10, K, 2)
    z = np.zeros_like(f["m"])
    a_q = A_of(oracle_mod, Q4_1, {"q": f["q"], "d": f["d"], "m": z}, x)
    a_m = A_of(oracle_mod, Q4_1, {"q": np.zeros_like(f["q"]), "d": f["d"], "m": f["m"]}, x)
    a_1 = A_of(oracle_mod, Q4_1, {"q": np.ones_like(f["q"]), "d": f["d"], "m": z}, x)
    for beta in (0, 128):
        F = F_of(oracle_mod, Q4_1, f, x, beta)
        assert np.allclose(F, a_q + a_m + 2 * beta * a_1, rtol=1e-12, atol=0), beta


def test_q4_k_against_condition_sums(oracle_mod):
    """d, dmin >= 0: F_beta = sum (d sc (q + 2 beta) + dmin m) |x|
    = A(codes q, m = 0) + A(codes 0: values -dmin m) + 2 beta A(codes 1, m = 0)."""
    f = fields(Q4_K, 11)
    x = synth.gen_x_seeded(12, K, 2)
    z = np.zeros_like(f["m"])
    base = {"sc": f["sc"], "d": f["d"], "dmin": f["dmin"]}
    a_q = A_of(oracle_mod, Q4_K, dict(base, q=f["q"], m=z), x)
    a_m = A_of(oracle_mod, Q4_K, dict(base, q=np.zeros_like(f["q"]), m=f["m"]), x)
    a_1 = A_of(oracle_mod, Q4_K, dict(base, q=np.ones_like(f["q"]), m=z), x)
    for beta in (0, 128):
        F = F_of(oracle_mod, Q4_K, f, x, beta)
        assert np.allclose(F, a_q + a_m + 2 * beta * a_1, rtol=1e-12, atol=0), beta


def test_q1_0_against_condition_sums(oracle_mod):
    """value = (2b - 1) d: s = 2d, q = b, mu = -d, so F_0 = sum d (2b + 1) |x|
    = 2 A(W, x masked to the elements with b = 1) + A(W, x)."""
    f = fields(Q1_0, 13)
    x = synth.gen_x_seeded(14, K, 1)
    W = synth.pack_fields(Q1_0, f)
    b = f["b"].reshape(M, K)
    F = F_of(oracle_mod, Q1_0, f, x, 0)
    A = A_of(oracle_mod, Q1_0, f, x)
    for r in range(M):
        xr = (x[0] * b[r]).astype(np.float32)[None, :]
        _, Ar, _ = oracle_mod.matvec(Q1_0, W, xr, M, K)
        assert np.isclose(F[0, r], 2 * Ar[0, r] + A[0, r], rtol=1e-12, atol=0), r


def test_q5_0_against_condition_sums(oracle_mod):
    """F_beta = sum |d| (q + 16 + 2 beta) |x| = A(codes q, as q5_1 with m = 0)
    + (16 + 2 beta) * A(codes 17, i.e. values d)."""
    f = fields(Q5_0, 15)
    x = synth.gen_x_seeded(16, K, 2)
    a_q = A_of(oracle_mod, Q5_1, {"q": f["q"], "d": f["d"], "m": np.zeros_like(f["d"])}, x)
    a_1 = A_of(oracle_mod, Q5_0, {"q": np.full_like(f["q"], 17), "d": f["d"]}, x)
    for beta in (0, 128):
        F = F_of(oracle_mod, Q5_0, f, x, beta)
        assert np.allclose(F, a_q + (16 + 2 * beta) * a_1, rtol=1e-12, atol=0), beta


def test_q6_k_against_condition_sums(oracle_mod):
    """mu = -32 s: F_beta = sum |s| (q + 32 + 2 beta) |x| = A(codes q + 32
    would overflow 6 bits, so): A(codes 33: values d sc) * (32 + 2 beta)
    + sum |s| q |x|, the last from the one-hot rows of x (F at x = e_k is the
    element's own |s| (q + 32 + 2 beta))."""
    f = fields(Q6_K, 17)
    x = synth.gen_x_seeded(18, K, 2)
    a_1 = A_of(oracle_mod, Q6_K, {"q": np.full_like(f["q"], 33), "sc": f["sc"], "d": f["d"]}, x)
    F0 = F_of(oracle_mod, Q6_K, f, x, 0)
    F128 = F_of(oracle_mod, Q6_K, f, x, 128)
    assert np.allclose(F128 - F0, 256 * a_1, rtol=1e-9, atol=0)
    # one-hot: element (r, k) alone; A there is |s| |q - 32|, F_0 is |s| (q + 32)
    W = synth.pack_fields(Q6_K, f)
    q = f["q"].reshape(M, K).astype(np.float64)
    for k in (0, 15, 16, 300, 511):
        e = np.zeros((1, K), np.float32)
        e[0, k] = 1.0
        _, A, F, _ = oracle_mod.matvec_f(Q6_K, W, e, M, K, 0)
        ok = q[:, k] != 32
        s = np.zeros(M)
        s[ok] = A[0][ok] / np.abs(q[ok, k] - 32)
        assert np.allclose(F[0][ok], s[ok] * (q[ok, k] + 32), rtol=1e-12, atol=0), k


@pytest.mark.parametrize("fmt", [Q5_K, Q2_K])
def test_k_quants_with_min_against_condition_sums(oracle_mod, fmt):
    """d, dmin >= 0: F_beta = A(codes q, m = 0) + A(codes 0: values -dmin m)
    + 2 beta A(codes 1, m = 0)."""
    f = fields(fmt, 19)
    x = synth.gen_x_seeded(20, K, 2)
    z = np.zeros_like(f["m"])
    base = {"sc": f["sc"], "d": f["d"], "dmin": f["dmin"]}
    a_q = A_of(oracle_mod, fmt, dict(base, q=f["q"], m=z), x)
    a_m = A_of(oracle_mod, fmt, dict(base, q=np.zeros_like(f["q"]), m=f["m"]), x)
    a_1 = A_of(oracle_mod, fmt, dict(base, q=np.ones_like(f["q"]), m=z), x)
    for beta in (0, 128):
        F = F_of(oracle_mod, fmt, f, x, beta)
        assert np.allclose(F, a_q + a_m + 2 * beta * a_1, rtol=1e-12, atol=0), beta


def test_q5_1_against_condition_sums(oracle_mod):
    f = fields(Q5_1, 21)
    assert (f["m"].astype(np.float64) <= 0).all()
    x = synth.gen_x_seeded(22, K, 2)
    z = np.zeros_like(f["m"])
    a_q = A_of(oracle_mod, Q5_1, {"q": f["q"], "d": f["d"], "m": z}, x)
    a_m = A_of(oracle_mod, Q5_1, {"q": np.zeros_like(f["q"]), "d": f["d"], "m": f["m"]}, x)
    a_1 = A_of(oracle_mod, Q5_1, {"q": np.ones_like(f["q"]), "d": f["d"], "m": z}, x)
    for beta in (0, 128):
        F = F_of(oracle_mod, Q5_1, f, x, beta)
        assert np.allclose(F, a_q + a_m + 2 * beta * a_1, rtol=1e-12, atol=0), beta
