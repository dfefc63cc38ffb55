"""lw_attn_decode against the oracle: one query token over a KV cache in each
cache format, grouped-query head ratios 1 to 8, head_dim 64 and 128, from
one cached position to tens of thousands (splits with a ragged last one),
peaked and flat softmax.

Bar (lw.h): |out - ref| <= 2^-12 * (1 + T) * A per output, A = sum_j p_j |v_j|
and T the head's largest scale * sum |q k|; NMSE against the paper's 1e-7."""
import numpy as np
import pytest

from gpu_util import to_gpu
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q4_0, Q4_1, Q5_0, Q5_1, Q8_0

pytestmark = pytest.mark.gpu

KV_FMTS = [F16, Q8_0, Q4_0, Q4_1, Q5_0, Q5_1, MXFP4]


def make(fmt, n_kv, L, D, seed, sigma=1.0):
    return synth.pack_fields(fmt, synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(seed), sigma))


def check(oracle_mod, fmt, q, Kc, Vc, H, n_kv, D, L, scale, what):
    import torch
    print("attn fmt=%d H=%d n_kv=%d D=%d L=%d" % (fmt, H, n_kv, D, L), flush=True)
    out = binding.attn_decode(fmt, to_gpu(q), to_gpu(Kc), to_gpu(Vc), H, n_kv, D, L, scale)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref, A, T = oracle_mod.attn_decode(fmt, q, Kc, Vc, H, n_kv, D, L, scale)
    err = np.abs(got - ref)
    bound = 2.0 ** -12 * (1 + T)[:, None] * A
    assert np.isfinite(got).all(), what
    assert (err <= bound).all(), (what, float((err / bound).max()))
    nmse = float((err ** 2).sum() / (ref ** 2).sum())
    assert nmse <= 1e-7, (what, nmse)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(bound > 0, err / bound, 0.0)
    return float(ratio.max()), nmse


@pytest.mark.parametrize("fmt", KV_FMTS)
@pytest.mark.parametrize("H,n_kv,D,L", [(32, 8, 128, 1), (32, 8, 128, 7), (32, 8, 128, 2048), (32, 8, 128, 5001),
                                        (8, 8, 64, 100), (16, 2, 64, 334), (64, 8, 128, 4096), (8, 1, 128, 66),
                                        (16, 8, 64, 40000)])
def test_attn_parity(oracle_mod, fmt, H, n_kv, D, L):
    Kc, Vc = make(fmt, n_kv, L, D, 1), make(fmt, n_kv, L, D, 2)
    q = np.random.default_rng([3, H, D]).standard_normal((H, D)).astype(np.float32)
    r, nmse = check(oracle_mod, fmt, q, Kc, Vc, H, n_kv, D, L, 1 / np.sqrt(D), (fmt, H, n_kv, D, L))
    print("  bound ratio %.3g NMSE %.3g" % (r, nmse), flush=True)


@pytest.mark.parametrize("fmt", [F16, Q8_0, Q4_0])
def test_attn_peaked_and_flat(oracle_mod, fmt):
    """Large logits (query scaled by 16: nearly one-hot weights) and a zero
    query (uniform weights over every position)."""
    H, n_kv, D, L = 32, 8, 128, 3000
    Kc, Vc = make(fmt, n_kv, L, D, 4), make(fmt, n_kv, L, D, 5)
    q = np.random.default_rng(6).standard_normal((H, D)).astype(np.float32)
    check(oracle_mod, fmt, (q * 16).astype(np.float32), Kc, Vc, H, n_kv, D, L, 1 / np.sqrt(D), "peaked")
    check(oracle_mod, fmt, np.zeros((H, D), np.float32), Kc, Vc, H, n_kv, D, L, 1 / np.sqrt(D), "flat")


MF_FMTS = [F16, Q8_0, Q4_0]


@pytest.mark.parametrize("fmt", MF_FMTS)
@pytest.mark.parametrize("H,n_kv,D,L", [(8, 8, 128, 2080), (16, 8, 128, 9000), (32, 8, 128, 12345),
                                        (64, 8, 128, 9000), (32, 8, 64, 9000), (64, 8, 64, 5000),
                                        (16, 2, 64, 20000), (4, 1, 128, 40000)])
def test_attn_matrix_core_scores(oracle_mod, fmt, H, n_kv, D, L):
    """The matrix-core score kernel (more than 64 positions per split) over
    every head ratio and head size: 65-position splits whose last tile holds
    one position, ragged last splits, one key/value head."""
    assert binding.attn_kernel_name(fmt, H, n_kv, D, L).startswith("attn_mf_kernel")
    Kc, Vc = make(fmt, n_kv, L, D, 21), make(fmt, n_kv, L, D, 22)
    q = np.random.default_rng([23, H, D]).standard_normal((H, D)).astype(np.float32)
    r, nmse = check(oracle_mod, fmt, q, Kc, Vc, H, n_kv, D, L, 1 / np.sqrt(D), (fmt, H, n_kv, D, L))
    print("  bound ratio %.3g NMSE %.3g" % (r, nmse), flush=True)


@pytest.mark.parametrize("fmt", MF_FMTS)
def test_attn_matrix_core_query_range(oracle_mod, fmt):
    """The query's per-head power-of-two scaling of the matrix-core kernel:
    queries scaled by 2^60 and 2^-60, one with elements spread over 2^-20 ..
    2^20 within a head, peaked and zero queries."""
    H, n_kv, D, L = 32, 8, 128, 9000
    assert binding.attn_kernel_name(fmt, H, n_kv, D, L).startswith("attn_mf_kernel")
    Kc, Vc = make(fmt, n_kv, L, D, 24), make(fmt, n_kv, L, D, 25)
    rng = np.random.default_rng(26)
    q = rng.standard_normal((H, D)).astype(np.float32)
    spread = (q * np.exp2(rng.integers(-20, 21, (H, D)))).astype(np.float32)
    sc = 1 / np.sqrt(D)
    check(oracle_mod, fmt, (q * 2.0 ** 60).astype(np.float32), Kc, Vc, H, n_kv, D, L, sc * 2.0 ** -60, "2^60")
    check(oracle_mod, fmt, (q * 2.0 ** -60).astype(np.float32), Kc, Vc, H, n_kv, D, L, sc * 2.0 ** 60, "2^-60")
    check(oracle_mod, fmt, spread, Kc, Vc, H, n_kv, D, L, sc * 2.0 ** -16, "spread")
    check(oracle_mod, fmt, (q * 16).astype(np.float32), Kc, Vc, H, n_kv, D, L, sc, "peaked")
    check(oracle_mod, fmt, np.zeros((H, D), np.float32), Kc, Vc, H, n_kv, D, L, sc, "flat")


# the code of an exact zero, per format with one
ZERO_CODE = {F16: ("w", 0), Q8_0: ("q", 0), Q4_0: ("q", 8), Q5_0: ("q", 16), MXFP4: ("q", 0)}


@pytest.mark.parametrize("fmt", sorted(ZERO_CODE))
@pytest.mark.parametrize("L", [1000, 9000])
def test_attn_zero_values_exact(oracle_mod, fmt, L):
    """A cache dimension whose values are all exactly zero (every position,
    every key/value head), and a key row of zeros: A = 0 for that output
    dimension, so the bound asks for an exact zero there. 1000 positions
    run the vector kernel for every format, 9000 the matrix-core score
    kernel for f16, Q8_0 and Q4_0."""
    H, n_kv, D = 32, 8, 128
    key, zero = ZERO_CODE[fmt]
    rng = np.random.default_rng([27, fmt, L])
    fk = synth.gen_fields_eq1(fmt, n_kv * L * D, rng, 1.0)
    fv = synth.gen_fields_eq1(fmt, n_kv * L * D, rng, 1.0)
    col = (np.arange(n_kv * L * D) % D) == 5
    fv[key][col] = zero
    fk[key][(np.arange(n_kv * L * D) // D) % L == 17] = zero  # position 17 of every head: k = 0
    Kc, Vc = synth.pack_fields(fmt, fk), synth.pack_fields(fmt, fv)
    q = rng.standard_normal((H, D)).astype(np.float32)
    check(oracle_mod, fmt, q, Kc, Vc, H, n_kv, D, L, 1 / np.sqrt(D), (fmt, L))
    out = binding.attn_decode(fmt, to_gpu(q), to_gpu(Kc), to_gpu(Vc), H, n_kv, D, L, 1 / np.sqrt(D))
    assert (out.cpu().numpy()[:, 5] == 0).all(), (fmt, L)


def test_attn_stream_and_workspace_reuse(oracle_mod):
    """Two calls on one stream sharing a workspace, the second smaller; each
    output matches the oracle."""
    import torch
    s = torch.cuda.Stream()
    ws = torch.empty(binding.attn_workspace_bytes(Q8_0, 32, 8, 128, 4096), dtype=torch.uint8, device="cuda")
    outs = []
    cases = [(4096, 11), (700, 12)]
    with torch.cuda.stream(s):
        for L, seed in cases:
            Kc, Vc = make(Q8_0, 8, L, 128, seed), make(Q8_0, 8, L, 128, seed + 100)
            q = np.random.default_rng(seed).standard_normal((32, 128)).astype(np.float32)
            o = binding.attn_decode(Q8_0, to_gpu(q), to_gpu(Kc), to_gpu(Vc), 32, 8, 128, L, 0.088, workspace=ws,
                                    stream=s)
            outs.append((o, q, Kc, Vc, L))
    s.synchronize()
    for o, q, Kc, Vc, L in outs:
        ref, A, T = oracle_mod.attn_decode(Q8_0, q, Kc, Vc, 32, 8, 128, L, 0.088)
        assert (np.abs(o.cpu().numpy() - ref) <= 2.0 ** -12 * (1 + T)[:, None] * A).all(), L
