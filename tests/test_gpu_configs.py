"""Parity at the full workload sizes, in the launch configuration the
benchmark times (one lw_matvec per matrix): the single Q8_0 matrix in full,
the other workloads on sampled outputs (first, last and random rows) that the
oracle computes one by one."""
import numpy as np
import pytest

import gate
from gpu_util import to_gpu
from paper_2605_20706_amd import binding, synth

pytestmark = pytest.mark.gpu


def sampled_rows(M, n_rand, seed):
    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([np.arange(min(8, M)), np.arange(max(0, M - 8), M),
                                     rng.integers(0, M, n_rand)]))
    return rows


def run(wl, mat, n_tok=1):
    import torch
    W = synth.gen_matrix(wl, mat)
    x = synth.gen_x(wl, mat.K, n_tok)
    y = binding.matvec(wl.fmt, to_gpu(W), to_gpu(x), mat.M, mat.K)
    torch.cuda.synchronize()
    return W, x, y.cpu().numpy()


def test_q8_0_2048_full(oracle_mod):
    wl = synth.WORKLOADS["q8_0_2048"]
    mat = wl.matrices[0]
    W, x, y = run(wl, mat)
    y_ref, A, _ = oracle_mod.matvec(wl.fmt, W, x, mat.M, mat.K)
    m = gate.check(y, y_ref, A, f32_bound=1e-4)
    print("q8_0_2048", m)


# one matrix of every distinct shape of each workload (layer 0, and the lm_head)
CASES = [("f16_llama1b", i) for i in range(5)] + [("q4_0_llama1b", i) for i in (0, 1, 2, 4, 80)] + \
        [("q4_k_llama8b", i) for i in (0, 1, 2, 4, 160)] + [("q4_0_llama8b_ffn", i) for i in range(3)] + \
        [("q4_1_llama8b_ffn", i) for i in range(3)] + [("q1_0_1b7", i) for i in (0, 1, 2, 4, 140)]


@pytest.mark.parametrize("key,idx", CASES)
def test_workload_matrix_sampled(oracle_mod, key, idx):
    wl = synth.WORKLOADS[key]
    mat = wl.matrices[idx]
    print("workload %s matrix %s %dx%d" % (key, mat.name, mat.M, mat.K), flush=True)
    W, x, y = run(wl, mat)
    rows = sampled_rows(mat.M, 48, idx)
    y_ref, A = oracle_mod.matvec_sampled(wl.fmt, W, x, mat.M, mat.K, rows, np.zeros_like(rows))
    gate.check(y[0, rows], y_ref, A, f32_bound=1e-4, what=(key, idx))


@pytest.mark.parametrize("key", ["q4_0_llama8b_ffn", "q4_1_llama8b_ffn"])
@pytest.mark.parametrize("idx", range(3))
def test_multi_token_ffn(oracle_mod, key, idx):
    """n_tok in {1, 2, 4, 8} and 512 on the 8B gate/up/down matrices; every
    token column of a batched call also agrees with its own n_tok = 1 call."""
    import torch
    wl = synth.WORKLOADS[key]
    mat = wl.matrices[idx]
    W = synth.gen_matrix(wl, mat)
    Wg = to_gpu(W)
    x = synth.gen_x(wl, mat.K, 512)
    xg = to_gpu(x)
    rows = sampled_rows(mat.M, 24, 100 + idx)
    singles = {}
    for nt in (1, 2, 4, 8, 512):
        print("ffn %s n_tok=%d" % (mat.name, nt), flush=True)
        y = binding.matvec(wl.fmt, Wg, xg[:nt], mat.M, mat.K)
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        if nt <= 8:
            toks = np.repeat(np.arange(nt), rows.size)
            rr = np.tile(rows, nt)
        else:
            rng = np.random.default_rng(idx)
            toks = np.concatenate([np.repeat([0, 511], rows.size), rng.integers(0, 512, 256)])
            rr = np.concatenate([rows, rows, rng.integers(0, mat.M, 256)])
        y_ref, A = oracle_mod.matvec_sampled(wl.fmt, W, x, mat.M, mat.K, rr, toks)
        gate.check(y[toks, rr], y_ref, A, f32_bound=1e-4 if nt <= 8 else None, what=(mat.name, nt))
        if nt == 1:
            singles[0] = y[0]
        else:
            d = np.abs(y[0].astype(np.float64) - singles[0]).max()
            assert d <= gate.TOL * np.abs(singles[0]).max(), (mat.name, nt, d)
