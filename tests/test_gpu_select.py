"""Every candidate of the kernel-selection table, forced through the
LW_FORCE_CFG override, against the oracle on shapes with ragged row groups:
a sweep may pick any of them, so each must meet the same bar as the built-in
choices (the float32 bound with the term mass of its form)."""
import os

import numpy as np
import pytest

import gate
from gpu_util import to_gpu
from parity import Ref, kernel_of
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import Q4_0, Q4_1, Q4_K

pytestmark = pytest.mark.gpu

REG1 = {10: 2048, 11: 2048, 12: 2048, 13: 4096, 14: 4096, 15: 4096, 16: 4096, 17: 4096, 18: 14336, 19: 14336,
        20: 14336}
REG2 = {21: 2048, 22: 4096, 23: 8192, 24: 14336, 25: 4096}
CASES = ([(c, K, 1, M) for c, K in REG1.items() for M in (17, 3001)]
         + [(c, K, 2, M) for c, K in REG2.items() for M in (5, 2500)]
         + [(1, 4096, 1, 3001), (30, 4096, 4, 8200), (31, 2304, 5, 300), (31, 2304, 12, 300),
            (32, 2304, 9, 300), (32, 4352, 16, 1100)])


class forced:
    def __init__(self, cand):
        self.cand = cand

    def __enter__(self):
        self.old = os.environ.get("LW_FORCE_CFG")
        os.environ["LW_FORCE_CFG"] = str(self.cand)

    def __exit__(self, *a):
        if self.old is None:
            del os.environ["LW_FORCE_CFG"]
        else:
            os.environ["LW_FORCE_CFG"] = self.old


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1])
@pytest.mark.parametrize("cand,K,n_tok,M", CASES)
def test_forced_candidate(oracle_mod, fmt, cand, K, n_tok, M):
    import torch
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([cand, fmt, M, K]))
    x = synth.gen_x_seeded([cand, K, n_tok], K, n_tok)
    with forced(cand):
        kern = kernel_of(fmt, M, K, n_tok)
        print("cand %d fmt=%d M=%d K=%d n_tok=%d -> %s" % (cand, fmt, M, K, n_tok, kern), flush=True)
        y = binding.matvec(fmt, to_gpu(W), to_gpu(x), M, K)
        torch.cuda.synchronize()
    ref = Ref(oracle_mod, fmt, W, x, M, K)
    gate.check(y.cpu().numpy(), ref.y, ref.A, ref.F(kern), f32_bound=1e-4, what=(cand, fmt, M, K, n_tok, kern))


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K])
@pytest.mark.parametrize("cand,K", [(c, K) for c, K in REG1.items()])
def test_forced_candidate_fused_pair(oracle_mod, fmt, cand, K):
    """The fused single-token launch of lw_matvec_multi over two matrices
    (a layer's gate and up) with each register candidate."""
    import torch
    Ms = [1500, 1001]
    Ws = [synth.gen_packed(fmt, m * K, np.random.default_rng([cand, fmt, i])) for i, m in enumerate(Ms)]
    x = synth.gen_x_seeded([cand, K], K, 1)
    with forced(cand):
        kern = kernel_of(fmt, Ms[0], K, 1, Ms=Ms)
        print("cand %d multi fmt=%d Ms=%s K=%d -> %s" % (cand, fmt, Ms, K, kern), flush=True)
        ys = binding.matvec_multi(fmt, [to_gpu(w) for w in Ws], to_gpu(x), Ms, K)
        torch.cuda.synchronize()
    for w, m, yg in zip(Ws, Ms, ys):
        ref = Ref(oracle_mod, fmt, w, x, m, K)
        gate.check(yg.cpu().numpy(), ref.y, ref.A, ref.F(kern), f32_bound=1e-4, what=(cand, fmt, m, K))
