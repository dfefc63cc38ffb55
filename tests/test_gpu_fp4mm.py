"""LW_MXFP4 prefill on the fp4 matrix cores (lw_matvec_ws) against the oracle.

Every output is compared, at sizes that span several row and token tiles
with ragged tails, the K-split launch (partial results added into a zeroed
y) and the unsplit one, the method's edge inputs, and the 8B FFN set at 512
tokens. Bar: the fp4 path's bound |y - y_ref| <= 2^-16 Bm + 2^-11 (A + Bm/4)
(tests/gate.py: the activations' split into four e2m3 pieces, then the
matrix core's own summation) and the 2e-3 normwise gate."""
import numpy as np
import pytest

import gate
from gpu_util import to_gpu
from parity import block_max_mass
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import MXFP4

pytestmark = pytest.mark.gpu

FP4_KERNEL = "fp4mm_kernel<"


def run_ws(fmt, W, x, M, K, ws=None):
    import torch
    y = binding.matvec_ws(fmt, to_gpu(W), to_gpu(np.atleast_2d(x)), M, K, workspace=ws)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check(oracle_mod, W, x, M, K, y, what):
    y_ref, A, _ = oracle_mod.matvec(MXFP4, W, x, M, K)
    Bm = block_max_mass(oracle_mod, MXFP4, W, x, M, K)
    m = gate.check_fp4(y, y_ref, A, Bm, what=what)
    print("  %s fp4_ratio=%.3g scaled=%.3g normwise=%.3g nmse=%.3g" % (what, m["fp4_ratio"], m["scaled"],
                                                                     m["normwise"], m["nmse"]), flush=True)
    return m


@pytest.mark.parametrize("M,K,n_tok", [
    (1100, 4352, 100),  # 3 x 2 tiles, ragged rows and tokens (K split: y zeroed, partials added)
    (300, 1024, 17),    # one tile, 17 tokens (the first count the path takes)
    (8192, 512, 240),   # 16 x 4 tiles, unsplit
    (41, 2048, 67),     # 41 rows: most of the row tile masked
    (513, 256, 129),    # odd M (scalar stores), the smallest K
    (4096, 4096, 64),   # one whole token tile, float4 stores
])
def test_fp4mm_tiles(oracle_mod, M, K, n_tok):
    W = synth.gen_packed(MXFP4, M * K, np.random.default_rng([80, M, K]))
    x = synth.gen_x_seeded([81, M, K], K, n_tok)
    assert binding.kernel_name_ws(MXFP4, M, K, n_tok).startswith(FP4_KERNEL)
    print("fp4mm M=%d K=%d n_tok=%d launches=%d" % (M, K, n_tok, binding.launch_count_ws(MXFP4, M, K, n_tok)),
          flush=True)
    y = run_ws(MXFP4, W, x, M, K)
    check(oracle_mod, W, x, M, K, y, (M, K, n_tok))


KINDS = ["zero_rows", "zero_scales", "eq1_normal", "x_times_2^60", "x_times_2^-60", "sparse_x"]


@pytest.mark.parametrize("kind", KINDS)
def test_fp4mm_edges(oracle_mod, kind):
    """Rows of all-zero codes (+0 and -0) give exactly 0 (every product is
    0); blocks with the smallest exponent (2^-127, subnormal products);
    Eq. (1)-encoded N(0, 0.02^2) weights; activations scaled by 2^+-60 (the
    split's scales move with them); activations that are zero except one
    value per 32-block (a block's max is its only value: the split is exact)."""
    M, K, n_tok = 1100, 2304, 70
    rng = np.random.default_rng([82, KINDS.index(kind)])
    zrows = None
    if kind == "zero_rows":
        f = synth.gen_fields_eq1(MXFP4, M * K, rng)
        zrows = np.unique(np.concatenate([[0, 1, M // 2, M - 1], rng.integers(0, M, M // 64)]))
        f = synth.zero_rows(MXFP4, f, zrows, K)
    elif kind == "zero_scales":
        f = synth.zero_scales(MXFP4, synth.gen_fields(MXFP4, M * K, rng), rng)
    elif kind == "eq1_normal":
        f = synth.gen_fields_eq1(MXFP4, M * K, rng)
    else:
        f = synth.gen_fields(MXFP4, M * K, rng)
    W = synth.pack_fields(MXFP4, f)
    x = synth.gen_x_seeded([83, KINDS.index(kind)], K, n_tok)
    if kind == "x_times_2^60":
        x = (x.astype(np.float64) * 2.0 ** 60).astype(np.float32)
    elif kind == "x_times_2^-60":
        x = (x.astype(np.float64) * 2.0 ** -60).astype(np.float32)
    elif kind == "sparse_x":
        keep = np.zeros_like(x, dtype=bool)
        keep.reshape(n_tok, K // 32, 32)[:, :, 0] = True
        x = np.where(keep, x, np.float32(0))
    y = run_ws(MXFP4, W, x, M, K)
    check(oracle_mod, W, x, M, K, y, (kind, M, K, n_tok))
    if zrows is not None:
        assert (y[:, zrows] == 0).all(), "rows of zero codes must give exactly 0"


def test_fp4mm_llama8b_ffn_every_output(oracle_mod):
    """The 8B FFN set (gate and up 14336 x 4096, down 4096 x 14336) at 512
    tokens, every output, with one workspace shared by the three calls."""
    import torch
    wl = synth.WORKLOADS["mxfp4_llama8b_ffn"]
    K0 = wl.matrices[0].K
    need = max(binding.matvec_workspace_bytes(MXFP4, m.M, m.K, 512) for m in wl.matrices)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    for mat in wl.matrices:
        W = synth.gen_matrix(wl, mat)
        x = synth.gen_x(wl, mat.K, 512)
        print("ffn %s %dx%d (K0 %d)" % (mat.name, mat.M, mat.K, K0), flush=True)
        y = run_ws(MXFP4, W, x, mat.M, mat.K, ws=ws)
        check(oracle_mod, W, x, mat.M, mat.K, y, (mat.name, mat.M, mat.K, 512))


def test_fp4mm_workspace_reuse_and_smaller_call(oracle_mod):
    """Two calls in a row on one workspace, the second smaller: nothing of the
    first call's pieces leaks into the second."""
    import torch
    big = (2048, 4096, 300)
    small = (700, 1024, 33)
    ws = torch.empty(binding.matvec_workspace_bytes(MXFP4, *big), dtype=torch.uint8, device="cuda")
    for (M, K, n_tok), seed in ((big, 84), (small, 85)):
        W = synth.gen_packed(MXFP4, M * K, np.random.default_rng([seed, M]))
        x = synth.gen_x_seeded([seed, K], K, n_tok)
        y = run_ws(MXFP4, W, x, M, K, ws=ws)
        check(oracle_mod, W, x, M, K, y, ("reuse", M, K, n_tok))


@pytest.mark.parametrize("fmt,n_tok", [(2, 100), (3, 4), (11, 16), (11, 1), (0, 20)])
def test_ws_entry_is_lw_matvec_elsewhere(fmt, n_tok):
    """Calls that take no workspace path: lw_matvec_ws (workspace NULL) gives
    lw_matvec's bits."""
    import torch
    M, K = 1100, 2048
    assert binding.matvec_workspace_bytes(fmt, M, K, n_tok) == 0
    assert binding.kernel_name_ws(fmt, M, K, n_tok) == binding.kernel_name(fmt, M, K, n_tok)
    W = to_gpu(synth.gen_packed(fmt, M * K, np.random.default_rng([86, fmt])))
    x = to_gpu(synth.gen_x_seeded([87, fmt], K, n_tok))
    a = binding.matvec(fmt, W, x, M, K)
    b = binding.matvec_ws(fmt, W, x, M, K)
    torch.cuda.synchronize()
    if binding.launch_count(fmt, M, K, n_tok) == 1 or "gemm" not in binding.kernel_name(fmt, M, K, n_tok):
        assert torch.equal(a, b)
    else:  # a K-split launch adds its partials in any order
        assert torch.allclose(a, b, rtol=1e-5, atol=1e-5)
