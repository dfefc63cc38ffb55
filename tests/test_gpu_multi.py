"""lw_matvec_multi against the oracle: several matrices sharing the same
activations, as one launch (one token: the single-token kernels over the
concatenated rows; 3 to 8 tokens: the few-token matrix-core kernel, each
workgroup on rows of one matrix) or as one lw_matvec per matrix. Every output
meets the same bar as lw_matvec's, and each equals the separate lw_matvec
result within the gate."""
import numpy as np
import pytest

import gate
from gpu_util import to_gpu
from parity import kernel_of, reference
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

pytestmark = pytest.mark.gpu


def run_multi(oracle_mod, fmt, Ms, K, n_tok, seed):
    import torch
    Wh = [synth.gen_packed(fmt, m * K, np.random.default_rng([seed, fmt, i, m, K])) for i, m in enumerate(Ms)]
    x = synth.gen_x_seeded([seed, fmt, K], K, n_tok)
    Wg = [to_gpu(w) for w in Wh]
    xg = to_gpu(x)
    print("matvec_multi fmt=%d Ms=%s K=%d n_tok=%d" % (fmt, Ms, K, n_tok), flush=True)
    ys = binding.matvec_multi(fmt, Wg, xg, Ms, K)
    singles = [binding.matvec(fmt, w, xg, m, K) for w, m in zip(Wg, Ms)]
    torch.cuda.synchronize()
    for i, (w, m) in enumerate(zip(Wh, Ms)):
        y = ys[i].cpu().numpy()
        kern = kernel_of(fmt, m, K, n_tok, Ms=Ms)
        y_ref, A, F = reference(oracle_mod, fmt, w, x, m, K, kern)
        gate.check(y, y_ref, A, F, f32_bound=1e-4, what=(fmt, Ms, K, n_tok, i, kern))
        # the fused and the separate call each meet the bound: they differ by at most twice it
        gate.check(y, singles[i].cpu().numpy().astype(np.float64), 2 * A, None if F is None else 2 * F,
                   f32_bound=1e-4, what=("vs single", i))


@pytest.mark.parametrize("fmt", [F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4])
@pytest.mark.parametrize("Ms,K", [((67, 130, 1), 2304), ((17, 5), 256), ((33, 40, 64, 3), 4352)])
def test_multi_small(oracle_mod, fmt, Ms, K):
    """Ragged row counts (one launch over the LDS single-token kernel), up to
    the four-matrix limit; 2, 12 and 33 tokens (register, many-token and
    prefill kernels) go matrix by matrix."""
    for n_tok in (1, 2, 12, 33):
        run_multi(oracle_mod, fmt, list(Ms), K, n_tok, 31)


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1, Q1_0])
@pytest.mark.parametrize("Ms,K", [((14336, 14336), 4096), ((8192, 8192), 2048), ((2000, 3000, 9000), 14336)])
def test_multi_register_kernel(oracle_mod, fmt, Ms, K):
    """The register-activation kernel over the rows of two or three matrices
    (the 8B and 1B gate/up pairs, as the benchmark's decode step calls them;
    segments that end inside a row group and inside a workgroup)."""
    run_multi(oracle_mod, fmt, list(Ms), K, 1, 32)


@pytest.mark.parametrize("fmt", [F16, Q8_0, Q1_0])
def test_multi_lds_kernel_full_size(oracle_mod, fmt):
    """The LDS single-token kernel over the 1B gate/up pair (8192 + 8192 rows,
    K = 2048), the fused call of the benchmark's f16 decode step."""
    run_multi(oracle_mod, fmt, [8192, 8192], 2048, 1, 33)


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4, Q1_0])
@pytest.mark.parametrize("Ms,K", [((14336, 14336), 4096), ((3000, 3000, 2048), 4096), ((40000, 37, 40000), 256),
                                  ((70000, 70000), 256)])
def test_multi_fewtok_kernel(oracle_mod, fmt, Ms, K):
    """The few-token kernel over two to four matrices in one launch: the 8B
    gate/up pair, ragged segments whose last workgroup is short, a segment
    smaller than one workgroup's rows, and two or three tiles per wave."""
    # two tokens are fused too where no register kernel takes them
    for n_tok in ((3, 8) if fmt in (Q4_0, Q4_K, Q4_1, Q1_0) else (2, 3, 8)):
        name = binding.kernel_name_multi(fmt, list(Ms), K, n_tok)
        assert name.startswith("fewtok_kernel<%d, " % fmt), name
        run_multi(oracle_mod, fmt, list(Ms), K, n_tok, 34)


def test_multi_in_graph(oracle_mod):
    """A fused call captured into a HIP graph (as the benchmark runs it):
    every replay rewrites all outputs with the eager call's values."""
    import torch
    fmt, K, Ms = Q4_K, 4096, [14336, 14336]
    Wg = [to_gpu(synth.gen_packed(fmt, m * K, np.random.default_rng([40, i]))) for i, m in enumerate(Ms)]
    xg = to_gpu(synth.gen_x_seeded(41, K))
    eager = [v.clone() for v in binding.matvec_multi(fmt, Wg, xg, Ms, K)]
    ys = [torch.empty((1, m), dtype=torch.float32, device="cuda") for m in Ms]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        binding.matvec_multi(fmt, Wg, xg, Ms, K, ys=ys, stream=s)
    torch.cuda.synchronize()
    for _ in range(3):
        for v in ys:
            v.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i in range(len(Ms)):
            assert torch.equal(ys[i], eager[i]), i
