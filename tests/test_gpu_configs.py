"""Parity at the full workload sizes, every output of every matrix, in the
launch configuration the benchmark times: one lw_matvec per matrix, a
layer's gate and up projections as one lw_matvec_multi call (the decode
step's fused launch), all outputs compared with the oracle under the gate and
the float32 bound (tests/gate.py), F the term mass of the form the selected
kernel evaluates.

Workloads: the single Q8_0 2048x2048 matrix; the Llama-3.2-1B-shaped f16 set
(80 matrices); the 1B Q4_0 set with its lm_head (81); the Llama-3-8B-shaped
Q4_K-style set with its lm_head (161, in five parts); the 8B Q4_0 and Q4_1
FFN sets at 1, 2, 4, 8 and 512 tokens, and the other formats' 8B FFN sets at
the same counts; the 1.7B q1_0 set (141, in two parts) and its first layer
at 2, 4, 8 and 512 tokens."""
import os

import numpy as np
import pytest

import gate
from gpu_util import to_gpu
from parity import Ref, beta_of, kernel_of
from paper_2605_20706_amd import binding, synth

pytestmark = pytest.mark.gpu

N_THREADS = min(16, int(os.environ.get("OMP_NUM_THREADS", "0")) or 16)


def calls_of(mats, idx):
    """The benchmark's calls over matrices idx: a layer's gate followed by its
    up projection (same K) is one fused call, every other matrix one call."""
    calls = []
    for i in idx:
        m = mats[i]
        prev = calls[-1] if calls else None
        if (m.name == "up" and prev and len(prev) == 1 and mats[prev[0]].name == "gate"
                and mats[prev[0]].layer == m.layer and mats[prev[0]].K == m.K):
            calls[-1] = (prev[0], i)
        else:
            calls.append((i,))
    return calls


def run_calls(oracle_mod, wl, idx, n_tok=1):
    import torch
    mats = wl.matrices
    xs = {}
    worst = {"scaled": 0.0, "f32_ratio": 0.0, "normwise": 0.0, "nmse": 0.0}
    n_out = 0
    for call in calls_of(mats, idx):
        ms = [mats[i] for i in call]
        K = ms[0].K
        if K not in xs:
            xs[K] = synth.gen_x(wl, K, n_tok)
        x = xs[K]
        Wh = [synth.gen_matrix(wl, m) for m in ms]
        Wg = [to_gpu(w) for w in Wh]
        xg = to_gpu(x)
        Ms = [m.M for m in ms]
        kern = kernel_of(wl.fmt, Ms[0], K, n_tok, Ms=Ms if len(ms) > 1 else None)
        kerns = [kernel_of(wl.fmt, mm.M, K, n_tok, Ms=Ms if len(ms) > 1 else None) for mm in ms]
        print("%s %s n_tok=%d kernel=%s" % (wl.key, "+".join("%s[%d]" % (m.name, m.layer) for m in ms), n_tok, kern),
              flush=True)
        if len(ms) > 1:
            ys = binding.matvec_multi(wl.fmt, Wg, xg, Ms, K)
        else:
            ys = [binding.matvec(wl.fmt, Wg[0], xg, Ms[0], K)]
        torch.cuda.synchronize()
        for w, m, yg, kern in zip(Wh, ms, ys, kerns):
            ref = Ref(oracle_mod, wl.fmt, w, x, m.M, K, betas=(beta_of(kern),), n_threads=N_THREADS)
            mm = gate.check(yg.cpu().numpy(), ref.y, ref.A, ref.F(kern), f32_bound=1e-4,
                            what=(wl.key, m.name, m.layer, n_tok, kern))
            for k in worst:
                worst[k] = max(worst[k], mm[k])
            n_out += mm["n"]
        del Wg, ys
    print("  %d outputs: worst scaled %.3g, f32-bound ratio %.3g, normwise %.3g, NMSE %.3g"
          % (n_out, worst["scaled"], worst["f32_ratio"], worst["normwise"], worst["nmse"]), flush=True)
    return n_out


def parts(n, k):
    """Matrix indices [0, n) in k contiguous parts."""
    return [list(range(n * i // k, n * (i + 1) // k)) for i in range(k)]


CASES = ([("q8_0_2048", p) for p in parts(1, 1)] + [("f16_llama1b", p) for p in parts(80, 2)]
         + [("q4_0_llama1b", p) for p in parts(81, 1)] + [("q4_k_llama8b", p) for p in parts(161, 5)]
         + [("q1_0_1b7", p) for p in parts(141, 2)])


@pytest.mark.parametrize("key,idx", CASES, ids=["%s[%d:%d]" % (k, p[0], p[-1] + 1) for k, p in CASES])
def test_workload_every_output(oracle_mod, key, idx):
    wl = synth.WORKLOADS[key]
    n = run_calls(oracle_mod, wl, idx)
    assert n == sum(wl.matrices[i].M for i in idx)


@pytest.mark.parametrize("key", ["q4_0_llama8b_ffn", "q4_1_llama8b_ffn", "q5_0_llama8b_ffn", "q5_1_llama8b_ffn",
                                 "q5_k_llama8b_ffn", "q6_k_llama8b_ffn", "q2_k_llama8b_ffn", "mxfp4_llama8b_ffn"])
@pytest.mark.parametrize("n_tok", [1, 2, 4, 8, 512])
def test_ffn_every_output(oracle_mod, key, n_tok):
    """The 8B gate, up and down matrices at every token count of the
    multi-token workload, prefill (512 tokens) included: every output."""
    wl = synth.WORKLOADS[key]
    n = run_calls(oracle_mod, wl, range(len(wl.matrices)), n_tok)
    assert n == n_tok * sum(m.M for m in wl.matrices)


@pytest.mark.parametrize("n_tok", [2, 4, 8, 512])
def test_q1_0_layer_tokens_every_output(oracle_mod, n_tok):
    """The 1.7B q1_0 set's first layer (qkv, o, gate + up fused, down) at the
    multi-token counts of the benchmark: the register kernel (2 tokens), the
    few-token matrix-core kernel (4, 8) and the tiled one (512); every output."""
    wl = synth.WORKLOADS["q1_0_1b7"]
    n = run_calls(oracle_mod, wl, range(5), n_tok)
    assert n == n_tok * sum(wl.matrices[i].M for i in range(5))


@pytest.mark.parametrize("key", ["q4_0_llama8b_ffn"])
def test_token_columns_match_single_token(oracle_mod, key):
    """Every token column of a batched call agrees with the same token alone
    within twice the float32 bound (each meets it against the oracle)."""
    import torch
    wl = synth.WORKLOADS[key]
    for mat in wl.matrices:
        W = to_gpu(synth.gen_matrix(wl, mat))
        x = synth.gen_x(wl, mat.K, 8)
        xg = to_gpu(x)
        ref = Ref(oracle_mod, wl.fmt, synth.gen_matrix(wl, mat), x, mat.M, mat.K, n_threads=N_THREADS)
        for nt in (2, 4, 8):
            yb = binding.matvec(wl.fmt, W, xg[:nt], mat.M, mat.K)
            torch.cuda.synchronize()
            for t in range(nt):
                y1 = binding.matvec(wl.fmt, W, xg[t:t + 1], mat.M, mat.K)
                torch.cuda.synchronize()
                F = ref.Fs[128][t] + ref.Fs[0][t]
                gate.check(yb[t].cpu().numpy(), y1[0].cpu().numpy().astype(np.float64), 2 * ref.A[t], F,
                           f32_bound=1e-4, what=(mat.name, nt, t))
