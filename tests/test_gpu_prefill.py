"""Prefill (more than 16 tokens; every quantized format) on the matrix
cores against the oracle: several row and token tiles with ragged tails, the
K-split launch (partial products added into a zeroed y) with an uneven last
split and a half coefficient window, and the unsplit launch.

Bar: the gate, and the float32 bound 1e-4 * sum |w*x| + 2^-17 * F (the
activations enter the matrix cores as a bf16 high/low pair, exact to 2^-17;
F the term mass of the biased-code form, tests/gate.py)."""
import numpy as np
import pytest

import gate
from gpu_util import gpu_matvec, to_gpu
from parity import reference
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

pytestmark = pytest.mark.gpu


def run(oracle_mod, fmt, M, K, n_tok, seed):
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([seed, fmt, M, K]))
    x = synth.gen_x_seeded([seed + 1, fmt, K], K, n_tok)
    kern = binding.kernel_name(fmt, M, K, n_tok)
    print("prefill fmt=%d M=%d K=%d n_tok=%d kernel=%s" % (fmt, M, K, n_tok, kern), flush=True)
    y = gpu_matvec(fmt, W, x, M, K, Wg=to_gpu(W))
    y_ref, A, F = reference(oracle_mod, fmt, W, x, M, K, kern)
    gate.check(y, y_ref, A, F, f32_bound=1e-4, what=(fmt, M, K, n_tok))


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1, Q8_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4, Q1_0])
@pytest.mark.parametrize("M,K,n_tok", [
    (1100, 4352, 100),  # 3 x 2 tiles (ragged rows and tokens); K split 5 + 5 + 5 + 2 super-blocks
    (300, 1024, 17),    # one tile, 17 tokens (one past the few-token paths); unsplit (4 super-blocks)
    (8192, 512, 240),   # 16 x 4 tiles of the 4-bit tile, unsplit (two super-blocks)
    (41, 2048, 67),     # 41 rows (most of the row tile masked); two K splits; y of 2747 floats (a fill tail)
])
def test_prefill_tiles(oracle_mod, fmt, M, K, n_tok):
    run(oracle_mod, fmt, M, K, n_tok, 50)


@pytest.mark.parametrize("fmt", [F16])
@pytest.mark.parametrize("M,K,n_tok", [(300, 2304, 517), (1, 256, 64)])
def test_token_blocks_one_launch(oracle_mod, fmt, M, K, n_tok):
    """f16 runs many tokens as blocks of the matrix-vector kernel, all whole
    blocks in one launch (grid.y = block) and the remaining tokens in one
    more: 517 tokens are 64 blocks of 8 plus 5; 64 tokens leave no
    remainder."""
    run(oracle_mod, fmt, M, K, n_tok, 70)


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K])
def test_prefill_repeat_equal(oracle_mod, fmt):
    """The unsplit launch writes y with plain stores: two calls give the same
    bits. The split launch adds partials in any order: two calls agree to the
    float32 rounding of those additions."""
    import torch
    for M, K, n_tok, exact in [(8192, 512, 240, True), (1100, 4352, 100, False)]:
        W = to_gpu(synth.gen_packed(fmt, M * K, np.random.default_rng([60, fmt, M])))
        x = to_gpu(synth.gen_x_seeded([61, fmt], K, n_tok))
        a = binding.matvec(fmt, W, x, M, K)
        b = binding.matvec(fmt, W, x, M, K)
        torch.cuda.synchronize()
        if exact:
            assert torch.equal(a, b), (M, K, n_tok)
        else:
            d = (a - b).abs().max().item()
            assert d <= 1e-5 * a.abs().max().item(), (M, K, n_tok, d)
