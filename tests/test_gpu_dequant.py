"""lw_dequant is bit-exact against the oracle (+0 and -0 compare equal) on
exhaustive field domains, fuzzed scales and config-shaped tensors."""
import numpy as np
import pytest

from gpu_util import gpu_dequant, same_bits_or_both_zero
from paper_2605_20706_amd import layout, synth
from paper_2605_20706_amd.layout import F16, Q1_0, Q4_0, Q4_1, Q4_K, Q8_0

pytestmark = pytest.mark.gpu


def finite_halves():
    h = np.arange(65536, dtype=np.uint16)
    return h[np.isfinite(h.view(np.float16))]


def check(oracle_mod, fmt, W, n):
    print("dequant fmt=%d n=%d" % (fmt, n), flush=True)
    got = gpu_dequant(fmt, W, n)
    ref = oracle_mod.dequant(fmt, W, n)
    ok = same_bits_or_both_zero(got, ref)
    assert ok.all(), (fmt, n, np.flatnonzero(~ok)[:8], got[~ok][:8], ref[~ok][:8])


def test_f16_every_pattern(oracle_mod):
    h = np.arange(65536, dtype=np.uint16)
    check(oracle_mod, F16, layout.pack_f16(h), h.size)


def test_q8_0_every_code_every_scale(oracle_mod):
    d = finite_halves()
    q = np.tile(np.arange(-128, 128, dtype=np.int16), d.size).astype(np.int8)
    check(oracle_mod, Q8_0, layout.pack_q8_0(q, np.repeat(d, 8)), q.size)


def test_q4_0_every_code_every_scale(oracle_mod):
    d = finite_halves()
    q = np.tile(np.concatenate([np.arange(16), np.arange(16)]).astype(np.uint8), d.size)
    check(oracle_mod, Q4_0, layout.pack_q4_0(q, d), q.size)


def test_q4_k_fuzz_all_finite_scales(oracle_mod):
    rng = np.random.default_rng(99)
    nsb = 1 << 14
    n = 256 * nsb
    fin = finite_halves()
    W = layout.pack_q4_k(rng.integers(0, 16, n, dtype=np.uint8), rng.integers(0, 64, n // 32, dtype=np.uint8),
                         rng.integers(0, 64, n // 32, dtype=np.uint8), rng.choice(fin, nsb), rng.choice(fin, nsb))
    check(oracle_mod, Q4_K, W, n)


def test_q4_k_tie_and_hand_values(oracle_mod):
    # the single-rounding tie of the golden file: d=0x5A4E dmin=0x2678 sc=2 m=6 q=12
    q = np.full(256, 12, np.uint8)
    sc = np.full(8, 2, np.uint8)
    m = np.full(8, 6, np.uint8)
    W = layout.pack_q4_k(q, sc, m, np.array([0x5A4E], np.uint16), np.array([0x2678], np.uint16))
    got = gpu_dequant(Q4_K, W, 256)
    assert (got.view(np.uint32) == 0x45974ECA).all()


def test_q4_1_every_scale(oracle_mod):
    """All 16 codes x every finite binary16 d, random finite binary16 mins."""
    d = finite_halves()
    d = np.concatenate([d, d[: (-d.size) % 8]])  # whole super-block multiples of groups
    m = np.random.default_rng(98).choice(finite_halves(), d.size)
    q = np.tile(np.concatenate([np.arange(16), np.arange(16)]).astype(np.uint8), d.size)
    check(oracle_mod, Q4_1, layout.pack_q4_1(q, d, m), q.size)


def test_q4_1_tie_hand_value():
    # the round-to-nearest-even tie of the golden file: q=13 d=0x5A4E m=0x2678
    q = np.full(256, 13, np.uint8)
    W = layout.pack_q4_1(q, np.full(8, 0x5A4E, np.uint16), np.full(8, 0x2678, np.uint16))
    got = gpu_dequant(Q4_1, W, 256)
    assert (got.view(np.uint32) == 0x4523EC68).all()


def test_q1_0_every_scale_and_signed_zero(oracle_mod):
    """Both codes x every finite binary16 d (one scale per 128 elements):
    +d or -d, bit for bit; a zero scale with code 0 gives -0."""
    d = finite_halves()
    d = np.concatenate([d, d[: (-d.size) % 2]])  # whole multiples of 256 elements
    b = np.random.default_rng(97).integers(0, 2, 128 * d.size).astype(np.uint8)
    b[0::128], b[1::128] = 0, 1
    W = layout.pack_q1_0(b, d)
    check(oracle_mod, Q1_0, W, b.size)
    got = gpu_dequant(Q1_0, layout.pack_q1_0(np.zeros(256, np.uint8), np.zeros(2, np.uint16)), 256)
    assert (got.view(np.uint32) == 0x80000000).all()


@pytest.mark.parametrize("n", [256, 512 + 256, 4096 * 3 + 256])
@pytest.mark.parametrize("fmt", [F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0])
def test_small_and_ragged(oracle_mod, fmt, n):
    check(oracle_mod, fmt, synth.gen_packed(fmt, n, np.random.default_rng(n + fmt)), n)


@pytest.mark.parametrize("key,idx", [("q8_0_2048", 0), ("f16_llama1b", 4), ("q4_0_llama1b", 80),
                                     ("q4_k_llama8b", 0), ("q4_0_llama8b_ffn", 2)])
def test_config_tensors(oracle_mod, key, idx):
    wl = synth.WORKLOADS[key]
    mat = wl.matrices[idx]
    check(oracle_mod, wl.fmt, synth.gen_matrix(wl, mat), mat.M * mat.K)
