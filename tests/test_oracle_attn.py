"""Pins of the oracle's decode attention over a quantized KV cache (one query
token; Sec. 3.2 attention with K and V dequantized on load, Sec. 3.3 the
dequantization routines reused for the KV cache).

Checked against numpy's float64 softmax attention over the oracle's own
(separately pinned) dequantized caches, and against what the definition
fixes: one cached position returns its value row exactly, a zero query
averages the value rows, a jointly permuted cache leaves the output
unchanged, the grouped-query head mapping, a dominant key selects its value
row, and A = sum p |v| equals the output where every value is positive."""
import numpy as np
import pytest

from paper_2605_20706_amd import synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q4_0, Q4_1, Q5_0, Q5_1, Q8_0

KV_FMTS = [F16, Q8_0, Q4_0, Q4_1, Q5_0, Q5_1, MXFP4]


def cache(fmt, n_kv, L, D, seed, sigma=1.0):
    f = synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(seed), sigma)
    return synth.pack_fields(fmt, f)


def deq(oracle_mod, fmt, C, n_kv, L, D):
    return oracle_mod.dequant(fmt, C, n_kv * L * D).astype(np.float64).reshape(n_kv, L, D)


@pytest.mark.parametrize("fmt", KV_FMTS)
@pytest.mark.parametrize("H,n_kv,D,L", [(8, 2, 64, 10), (4, 4, 32, 3), (32, 8, 128, 40), (6, 1, 64, 1)])
def test_brute_force_vs_numpy(oracle_mod, fmt, H, n_kv, D, L):
    Kc, Vc = cache(fmt, n_kv, L, D, 1), cache(fmt, n_kv, L, D, 2)
    q = np.random.default_rng(3).standard_normal((H, D)).astype(np.float32)
    scale = 1.0 / np.sqrt(D)
    out, A, T = oracle_mod.attn_decode(fmt, q, Kc, Vc, H, n_kv, D, L, scale)
    Kd, Vd = deq(oracle_mod, fmt, Kc, n_kv, L, D), deq(oracle_mod, fmt, Vc, n_kv, L, D)
    g = np.arange(H) // (H // n_kv)
    s = np.einsum("hd,hjd->hj", q.astype(np.float64), Kd[g]) * scale
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    ref = np.einsum("hj,hjd->hd", p, Vd[g])
    refA = np.einsum("hj,hjd->hd", p, np.abs(Vd[g]))
    refT = (np.abs(q.astype(np.float64))[:, None, :] * np.abs(Kd[g])).sum(axis=2).max(axis=1) * scale
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-12 * np.abs(refA).max())
    assert np.allclose(A, refA, rtol=1e-12)
    assert np.allclose(T, refT, rtol=1e-12)


@pytest.mark.parametrize("fmt", KV_FMTS)
def test_single_position_returns_value_row(oracle_mod, fmt):
    H, n_kv, D = 8, 4, 64
    Kc, Vc = cache(fmt, n_kv, 2, D, 4), cache(fmt, n_kv, 2, D, 5)
    # a cache of two positions whose first position alone is attended: use kv_len = 1 over the
    # first n_kv * 1 * D elements, packed on their own
    Kc1, Vc1 = cache(fmt, n_kv, 1, D, 6), cache(fmt, n_kv, 1, D, 7)
    q = np.random.default_rng(8).standard_normal((H, D)).astype(np.float32)
    out, _, _ = oracle_mod.attn_decode(fmt, q, Kc1, Vc1, H, n_kv, D, 1, 0.125)
    Vd = deq(oracle_mod, fmt, Vc1, n_kv, 1, D)
    assert np.array_equal(out, Vd[np.arange(H) // 2, 0])
    del Kc, Vc


@pytest.mark.parametrize("fmt", KV_FMTS)
def test_zero_query_averages_values(oracle_mod, fmt):
    H, n_kv, D, L = 4, 2, 64, 37
    Kc, Vc = cache(fmt, n_kv, L, D, 9), cache(fmt, n_kv, L, D, 10)
    out, _, T = oracle_mod.attn_decode(fmt, np.zeros((H, D), np.float32), Kc, Vc, H, n_kv, D, L, 0.125)
    Vd = deq(oracle_mod, fmt, Vc, n_kv, L, D)
    assert np.allclose(out, Vd[np.arange(H) // 2].mean(axis=1), rtol=1e-13, atol=1e-15)
    assert (T == 0).all()


def test_joint_permutation_of_positions(oracle_mod):
    fmt, H, n_kv, D, L = Q8_0, 8, 2, 64, 24
    f_k = synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(11), 1.0)
    f_v = synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(12), 1.0)
    perm = np.random.default_rng(13).permutation(L)

    def permute(f):
        # rows of D elements = D/32 blocks each; codes and scales move with their row
        q = f["q"].reshape(n_kv, L, D)[:, perm].reshape(-1)
        d = f["d"].reshape(n_kv, L, D // 32)[:, perm].reshape(-1)
        return {"q": q, "d": d}
    q = np.random.default_rng(14).standard_normal((H, D)).astype(np.float32)
    a, _, _ = oracle_mod.attn_decode(fmt, q, synth.pack_fields(fmt, f_k), synth.pack_fields(fmt, f_v), H, n_kv, D, L,
                                     0.125)
    b, _, _ = oracle_mod.attn_decode(fmt, q, synth.pack_fields(fmt, permute(f_k)), synth.pack_fields(fmt, permute(f_v)),
                                     H, n_kv, D, L, 0.125)
    assert np.allclose(a, b, rtol=1e-13, atol=1e-15)


def test_grouped_query_heads(oracle_mod):
    """Heads of one group with the same query agree exactly; with as many
    key/value heads as query heads every head reads its own cache slice."""
    fmt, n_kv, D, L = Q4_0, 2, 64, 16
    Kc, Vc = cache(fmt, n_kv, L, D, 15), cache(fmt, n_kv, L, D, 16)
    q1 = np.random.default_rng(17).standard_normal(D).astype(np.float32)
    q = np.stack([q1] * 4 + [-q1] * 4)
    out, _, _ = oracle_mod.attn_decode(fmt, q, Kc, Vc, 8, n_kv, D, L, 0.125)
    for h in range(1, 4):
        assert np.array_equal(out[h], out[0]) and np.array_equal(out[4 + h], out[4])
    assert not np.array_equal(out[0], out[4])
    # two heads over two key/value heads: swapping the heads' cache slices swaps the outputs
    fk = synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(15), 1.0)
    fv = synth.gen_fields_eq1(fmt, n_kv * L * D, np.random.default_rng(16), 1.0)

    def swap(f):
        return {"q": np.concatenate(np.split(f["q"], 2)[::-1]), "d": np.concatenate(np.split(f["d"], 2)[::-1])}
    q2 = np.random.default_rng(18).standard_normal((2, D)).astype(np.float32)
    a, _, _ = oracle_mod.attn_decode(fmt, q2, synth.pack_fields(fmt, fk), synth.pack_fields(fmt, fv), 2, 2, D, L, 0.125)
    b, _, _ = oracle_mod.attn_decode(fmt, q2[::-1].copy(), synth.pack_fields(fmt, swap(fk)),
                                     synth.pack_fields(fmt, swap(fv)), 2, 2, D, L, 0.125)
    assert np.array_equal(a, b[::-1])
    del Kc, Vc


def test_dominant_key_selects_its_value(oracle_mod):
    fmt, H, n_kv, D, L = F16, 1, 1, 64, 9
    rng = np.random.default_rng(19)
    k = rng.standard_normal((L, D)).astype(np.float16)
    v = rng.standard_normal((L, D)).astype(np.float16)
    q = (k[5].astype(np.float32) * 40.0)[None, :]
    out, _, _ = oracle_mod.attn_decode(fmt, q, synth.pack_fields(F16, {"w": k.reshape(-1)}),
                                       synth.pack_fields(F16, {"w": v.reshape(-1)}), H, n_kv, D, L, 1.0)
    assert np.allclose(out[0], v[5].astype(np.float64), rtol=0, atol=1e-12)


def test_condition_sum_equals_output_for_positive_values(oracle_mod):
    fmt, H, n_kv, D, L = F16, 4, 2, 64, 20
    rng = np.random.default_rng(20)
    k = rng.standard_normal(n_kv * L * D).astype(np.float16)
    v = np.abs(rng.standard_normal(n_kv * L * D)).astype(np.float16) + np.float16(0.01)
    q = rng.standard_normal((H, D)).astype(np.float32)
    out, A, _ = oracle_mod.attn_decode(fmt, q, synth.pack_fields(F16, {"w": k}), synth.pack_fields(F16, {"w": v}),
                                       H, n_kv, D, L, 0.125)
    assert np.allclose(out, A, rtol=1e-14)


def test_rejects_bad_arguments(oracle_mod):
    C = cache(Q8_0, 2, 4, 64, 21)
    q = np.zeros((6, 64), np.float32)
    with pytest.raises(ValueError):
        oracle_mod.attn_decode(Q8_0, q, C, C, 6, 4, 64, 4, 0.1)   # 6 heads over 4 kv heads
    with pytest.raises(ValueError):
        oracle_mod.attn_decode(Q8_0, q[:, :48], C, C, 6, 2, 48, 4, 0.1)   # head_dim not whole blocks
