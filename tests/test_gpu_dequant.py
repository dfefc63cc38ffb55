"""lw_dequant is bit-exact against the oracle (+0 and -0 compare equal) on
exhaustive field domains, fuzzed scales and config-shaped tensors."""
import numpy as np
import pytest

from gpu_util import gpu_dequant, same_bits_or_both_zero
from paper_2605_20706_amd import layout, synth
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

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
@pytest.mark.parametrize("fmt", [F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4])
def test_small_and_ragged(oracle_mod, fmt, n):
    check(oracle_mod, fmt, synth.gen_packed(fmt, n, np.random.default_rng(n + fmt)), n)


@pytest.mark.parametrize("key,idx", [("q8_0_2048", 0), ("f16_llama1b", 4), ("q4_0_llama1b", 80),
                                     ("q4_k_llama8b", 0), ("q4_0_llama8b_ffn", 2)])
def test_config_tensors(oracle_mod, key, idx):
    wl = synth.WORKLOADS[key]
    mat = wl.matrices[idx]
    check(oracle_mod, wl.fmt, synth.gen_matrix(wl, mat), mat.M * mat.K)


def test_q5_0_every_code_every_scale(oracle_mod):
    d = finite_halves()
    q = np.tile(np.arange(32, dtype=np.uint8), d.size)
    check(oracle_mod, Q5_0, layout.pack_q5_0(q, d), q.size)


def test_q5_1_every_scale_and_tie(oracle_mod):
    d = finite_halves()
    m = np.random.default_rng(96).choice(finite_halves(), d.size)
    q = np.tile(np.arange(32, dtype=np.uint8), d.size)
    check(oracle_mod, Q5_1, layout.pack_q5_1(q, d, m), q.size)
    # the golden file's tie: q=17 d=0x5A4E m=0x2678 -> 0x45565C68
    W = layout.pack_q5_1(np.full(256, 17, np.uint8), np.full(8, 0x5A4E, np.uint16), np.full(8, 0x2678, np.uint16))
    assert (gpu_dequant(Q5_1, W, 256).view(np.uint32) == 0x45565C68).all()


@pytest.mark.parametrize("fmt", [Q5_K, Q2_K])
def test_k_quants_fuzz_all_finite_scales(oracle_mod, fmt):
    rng = np.random.default_rng(95 + fmt)
    nsb = 1 << 14
    n = 256 * nsb
    fin = finite_halves()
    per = 32 if fmt == Q5_K else 16
    top = 64 if fmt == Q5_K else 16
    q = rng.integers(0, 32 if fmt == Q5_K else 4, n, dtype=np.uint8)
    sc = rng.integers(0, top, n // per, dtype=np.uint8)
    m = rng.integers(0, top, n // per, dtype=np.uint8)
    pack = layout.pack_q5_k if fmt == Q5_K else layout.pack_q2_k
    check(oracle_mod, fmt, pack(q, sc, m, rng.choice(fin, nsb), rng.choice(fin, nsb)), n)


def test_k_quant_ties(oracle_mod):
    # golden ties: q5_k q=17 sc=2 m=6 d=0x5A4E dmin=0x2678 -> 0x45D65ACA;
    # q2_k q=1 sc=11 m=1 d=0x5A4E dmin=0x2678 -> 0x450AB398
    W = layout.pack_q5_k(np.full(256, 17, np.uint8), np.full(8, 2, np.uint8), np.full(8, 6, np.uint8),
                         np.array([0x5A4E], np.uint16), np.array([0x2678], np.uint16))
    assert (gpu_dequant(Q5_K, W, 256).view(np.uint32) == 0x45D65ACA).all()
    W = layout.pack_q2_k(np.full(256, 1, np.uint8), np.full(16, 11, np.uint8), np.full(16, 1, np.uint8),
                         np.array([0x5A4E], np.uint16), np.array([0x2678], np.uint16))
    assert (gpu_dequant(Q2_K, W, 256).view(np.uint32) == 0x450AB398).all()


def test_q6_k_every_code_every_scale(oracle_mod):
    """Every 6-bit code x every int8 scale (three d, one subnormal) and every
    finite binary16 d for one code and scale: exact values."""
    for dbits in (0x3C00, 0x2E66, 0x0003):
        q = np.tile(np.arange(64, dtype=np.uint8), 256 * 16)
        n = q.size
        sc = np.resize(np.repeat(np.arange(-128, 128, dtype=np.int16), 4).astype(np.int8), n // 16)
        check(oracle_mod, Q6_K, layout.pack_q6_k(q, sc, np.full(n // 256, dbits, np.uint16)), n)
    d = finite_halves()
    d = np.concatenate([d, d[: (-d.size) % 8]])
    rng = np.random.default_rng(94)
    q = rng.integers(0, 64, 256 * d.size, dtype=np.uint8)
    sc = rng.integers(-128, 128, 16 * d.size).astype(np.int8)
    check(oracle_mod, Q6_K, layout.pack_q6_k(q, sc, d), q.size)


def test_mxfp4_every_code_every_exponent(oracle_mod):
    """16 codes x all 256 e8m0 exponents: subnormal scales, overflow to
    infinity and the NaN exponent, bit for bit (NaN for NaN)."""
    E = np.arange(256).astype(np.uint8)
    codes = np.tile(np.concatenate([np.arange(16), np.arange(16)]).astype(np.uint8), E.size)
    check(oracle_mod, MXFP4, layout.pack_mxfp4(codes, E), codes.size)
