"""lw_matvec against the oracle on shapes spanning several 1 KiB chunks,
ragged row and column tails and every token count of the matrix-vector path,
plus token counts of the prefill path.

Bar: the gate (scaled error and normwise error <= 2e-3); every output must
also stay within the float32 bound 1e-4 * sum |w*x| + 2^-17 * F, F the term
mass of the factored form the selected kernel evaluates (tests/gate.py), far
below what any reduced-precision shortcut would give."""
import numpy as np
import pytest

import gate
from gpu_util import gpu_matvec, to_gpu
from parity import Ref, kernel_of, reference
from paper_2605_20706_amd import binding, synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

pytestmark = pytest.mark.gpu

FMTS = [F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4]
# (M, K): single row; row tail below a workgroup's rows; K below one chunk;
# K one chunk plus a ragged tail; several chunks; large K that needs x tiling.
SHAPES = [(1, 256), (3, 768), (17, 2048), (67, 2304), (130, 4352), (33, 16640)]
NTOKS = [1, 2, 3, 5, 8, 9, 16, 33]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,K", SHAPES)
def test_parity_small(oracle_mod, fmt, M, K):
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([fmt, M, K]))
    x = synth.gen_x_seeded([7, fmt, M, K], K, max(NTOKS))
    Wg = to_gpu(W)
    ref = Ref(oracle_mod, fmt, W, x, M, K)
    for nt in NTOKS:
        print("matvec fmt=%d M=%d K=%d n_tok=%d" % (fmt, M, K, nt), flush=True)
        y = gpu_matvec(fmt, W, x[:nt], M, K, Wg=Wg)
        kern = kernel_of(fmt, M, K, nt)
        gate.check(y, ref.y[:nt], ref.A[:nt], ref.F(kern, nt), f32_bound=1e-4, what=(fmt, M, K, nt, kern))


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1])
def test_parity_many_rows(oracle_mod, fmt):
    """Enough rows for the matrix-core few-token kernel to take two row groups
    per workgroup and four waves (a ragged last workgroup of one row group,
    K steps split unevenly over the waves)."""
    M, K = 16400, 1280
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([11, fmt]))
    x = synth.gen_x_seeded([12, fmt], K, 16)
    Wg = to_gpu(W)
    ref = Ref(oracle_mod, fmt, W, x, M, K)
    for nt in [2, 4, 7, 12, 13, 16]:
        print("matvec fmt=%d M=%d K=%d n_tok=%d" % (fmt, M, K, nt), flush=True)
        y = gpu_matvec(fmt, W, x[:nt], M, K, Wg=Wg)
        kern = kernel_of(fmt, M, K, nt)
        gate.check(y, ref.y[:nt], ref.A[:nt], ref.F(kern, nt), f32_bound=1e-4, what=(fmt, M, K, nt, kern))


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4, Q1_0])
@pytest.mark.parametrize("M,K", [(70000, 512), (300000, 256), (8200, 14336)])
def test_parity_few_tokens_tiles(oracle_mod, fmt, M, K):
    """Few-token matrix-core kernel with the activations in LDS: more 16-row
    tiles per workgroup than waves (two and four tiles per wave, a ragged last
    workgroup; the 5-bit formats at most two, their row groups capped), and
    three tiles per workgroup with a long K that takes four activation
    windows (the last one partial), each split over four waves."""
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([fmt, M, K, 21]))
    Wg = to_gpu(W)
    x = synth.gen_x_seeded([22, fmt, M, K], K, 8)
    ref = Ref(oracle_mod, fmt, W, x, M, K)
    for nt in (2, 3, 6, 8):
        print("matvec fmt=%d M=%d K=%d n_tok=%d" % (fmt, M, K, nt), flush=True)
        y = gpu_matvec(fmt, W, x[:nt], M, K, Wg=Wg)
        kern = kernel_of(fmt, M, K, nt)
        gate.check(y, ref.y[:nt], ref.A[:nt], ref.F(kern, nt), f32_bound=1e-4, what=(fmt, M, K, nt, kern))


# One to four tokens (the register kernel takes one or two, the matrix-core
# kernel more) over the 4-bit formats with K a whole number of
# 2048-element chunks (1, 2, 4 or 7 chunks per row): row counts from a single
# row to enough rows that every wave runs several full rounds of its row
# ring, with ragged row groups at the end.
REG_SHAPES = [(1, 2048), (40000, 2048), (9, 4096), (16500, 4096), (5, 8192), (8300, 8192),
              (1, 14336), (3500, 14336)]


@pytest.mark.parametrize("fmt", [Q4_0, Q4_K, Q4_1, Q1_0])
@pytest.mark.parametrize("M,K", REG_SHAPES)
def test_parity_whole_chunks(oracle_mod, fmt, M, K):
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([fmt, M, K, 5]))
    Wg = to_gpu(W)
    x = synth.gen_x_seeded([13, fmt, M, K], K, 4)
    ref = Ref(oracle_mod, fmt, W, x, M, K)
    for nt in (1, 2, 3, 4):
        print("matvec fmt=%d M=%d K=%d n_tok=%d" % (fmt, M, K, nt), flush=True)
        y = gpu_matvec(fmt, W, x[:nt], M, K, Wg=Wg)
        kern = kernel_of(fmt, M, K, nt)
        gate.check(y, ref.y[:nt], ref.A[:nt], ref.F(kern, nt), f32_bound=1e-4, what=(fmt, M, K, nt, kern))


@pytest.mark.parametrize("fmt", FMTS)
def test_one_hot_columns(oracle_mod, fmt):
    """x = e_k returns column k of the dequantized matrix: bit-exactly on the
    single-token path (one float32 product per output), within 1e-6 of the
    column magnitude when several one-hot tokens go through the matrix cores."""
    M, K = 70, 2304
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([3, fmt]))
    Wd = oracle_mod.dequant(fmt, W, M * K).reshape(M, K)
    Wg = to_gpu(W)
    ks = [0, 31, 32, 1000, 2047, 2048, 2303]
    x = np.zeros((len(ks), K), np.float32)
    for i, k in enumerate(ks):
        x[i, k] = 1.0
    for i, k in enumerate(ks):
        y1 = gpu_matvec(fmt, W, x[i], M, K, Wg=Wg)
        assert np.array_equal(y1[0], Wd[:, k]), (fmt, k)
    y = gpu_matvec(fmt, W, x, M, K, Wg=Wg)
    for i, k in enumerate(ks):
        err = np.abs(y[i].astype(np.float64) - Wd[:, k]).max()
        assert err <= 1e-6 * np.abs(Wd[:, k]).max(), (fmt, k, err)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("K", [2048, 2304])
def test_one_hot_every_lane_position(oracle_mod, fmt, K):
    """x = e_k for every element position k of two lanes' 32-element slices
    (and the last two of the row) returns column k of the dequantized matrix
    bit-exactly, on the register kernel (K = 2048) and the LDS kernel
    (K = 2304): pins the per-position handling of the one-token dots,
    including the 1- and 2-bit dots that pre-scale x by the power of two of
    each code's bit position."""
    M = 70
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([4, fmt, K]))
    Wd = oracle_mod.dequant(fmt, W, M * K).reshape(M, K)
    Wg = to_gpu(W)
    print("one-hot fmt=%d K=%d kernel=%s" % (fmt, K, binding.kernel_name(fmt, M, K, 1)), flush=True)
    for k in list(range(64)) + [K - 2, K - 1]:
        x = np.zeros(K, np.float32)
        x[k] = 1.0
        y = gpu_matvec(fmt, W, x, M, K, Wg=Wg)
        assert np.array_equal(y[0], Wd[:, k]), (fmt, K, k)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("n_tok", [1, 2, 4, 12, 33])
def test_zero_x_gives_exact_zero(oracle_mod, fmt, n_tok):
    """x = 0: every sum a kernel forms is a sum of zeros, so y is exactly 0 on
    every path (zero weights with nonzero scales: tests/test_gpu_edges.py)."""
    M, K = 20, 512
    W = synth.gen_packed(fmt, M * K, np.random.default_rng([4, fmt]))
    y = gpu_matvec(fmt, W, np.zeros((n_tok, K), np.float32), M, K)
    assert (y == 0).all()


def test_y_is_overwritten(oracle_mod):
    import torch
    from paper_2605_20706_amd import binding
    M, K = 40, 1024
    W = synth.gen_packed(Q4_0, M * K, np.random.default_rng(5))
    x = synth.gen_x_seeded(6, K, 2)
    y = torch.full((2, M), float("nan"), device="cuda")
    binding.matvec(Q4_0, to_gpu(W), to_gpu(x), M, K, y=y)
    torch.cuda.synchronize()
    y_ref, A, F = reference(oracle_mod, Q4_0, W, x, M, K, kernel_of(Q4_0, M, K, 2))
    gate.check(y.cpu().numpy(), y_ref, A, F, f32_bound=1e-4)


def test_stream_argument(oracle_mod):
    """The call is enqueued on the given stream."""
    import torch
    from paper_2605_20706_amd import binding
    M, K = 64, 2048
    W = synth.gen_packed(Q4_K, M * K, np.random.default_rng(8))
    x = synth.gen_x_seeded(9, K)
    s = torch.cuda.Stream()
    Wg, xg = to_gpu(W), to_gpu(x)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        y = binding.matvec(Q4_K, Wg, xg, M, K, stream=s)
    s.synchronize()
    y_ref, A, F = reference(oracle_mod, Q4_K, W, x, M, K, kernel_of(Q4_K, M, K, 1))
    gate.check(y.cpu().numpy(), y_ref, A, F, f32_bound=1e-4)
