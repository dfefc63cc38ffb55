"""Pins of the oracle's dequantization against values fixed outside it.

Each test checks the oracle (plain C, ``oracle/lw_oracle.c``) against
something other than itself: numpy's binary16 conversion (a library routine),
exact double arithmetic on the drawn fields, hand-derived values and bytes in
``tests/golden/`` (each derived in its file from Eq. (1) of Sec. 2.2 and the
block structures of Sec. 2.2), and hand-built byte strings that fix the nibble
order and the scale-record bit positions independently of the packers.
"""
import numpy as np
import pytest

import golden_io
from paper_2605_20706_amd import layout
from paper_2605_20706_amd.layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0

FMT = {"f16": F16, "q8_0": Q8_0, "q4_0": Q4_0, "q4_k": Q4_K, "q4_1": Q4_1, "q1_0": Q1_0,
       "q5_0": Q5_0, "q5_1": Q5_1, "q5_k": Q5_K, "q6_k": Q6_K, "q2_k": Q2_K, "mxfp4": MXFP4}


def bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def same_bits_or_both_zero(a, b):
    """Bit-exact, except that +0 and -0 are equal."""
    a, b = np.asarray(a, np.float32), np.asarray(b, np.float32)
    return (bits(a) == bits(b)) | ((a == 0) & (b == 0))


def finite_halves():
    h = np.arange(65536, dtype=np.uint16)
    return h[np.isfinite(h.view(np.float16))]


# --------------------------------------------------------------------------- plane layout

def test_plane_sizes_golden(oracle_mod):
    for name, n, o1, o2, total in golden_io.plane_sizes():
        assert oracle_mod.weight_bytes(FMT[name], n) == total, name
        offs, tot = layout.plane_offsets(FMT[name], n)
        assert (offs[1], offs[2], tot) == (o1, o2, total), name


# --------------------------------------------------------------------------- f16

def test_f16_exhaustive_vs_numpy(oracle_mod):
    """All 65,536 binary16 patterns against numpy's float16 -> float32."""
    h = np.arange(65536, dtype=np.uint16)
    got = oracle_mod.dequant(F16, layout.pack_f16(h), h.size)
    ref = h.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(bits(got)[~nan], bits(ref)[~nan])  # sign of zero included
    # subnormals survive: 0x0001 is 2^-24
    assert got[1] == np.float32(2.0 ** -24)


# --------------------------------------------------------------------------- q8_0

@pytest.mark.slow
def test_q8_0_exhaustive(oracle_mod):
    """All 256 codes x every finite binary16 scale against exact double products."""
    d = finite_halves()                               # 63,488 scales
    q = np.tile(np.arange(-128, 128, dtype=np.int16), d.size).astype(np.int8)  # 8 groups per d
    dd = np.repeat(d, 8)
    got = oracle_mod.dequant(Q8_0, layout.pack_q8_0(q, dd), q.size)
    ref = (q.astype(np.float64) * np.repeat(d.view(np.float16).astype(np.float64), 256)).astype(np.float32)
    assert same_bits_or_both_zero(got, ref).all()


def test_q4_0_exhaustive(oracle_mod):
    """All 16 codes x every finite binary16 scale."""
    d = finite_halves()
    q = np.tile(np.concatenate([np.arange(16), np.arange(16)]).astype(np.uint8), d.size)
    got = oracle_mod.dequant(Q4_0, layout.pack_q4_0(q, d), q.size)
    ref = ((q.astype(np.float64) - 8.0) * np.repeat(d.view(np.float16).astype(np.float64), 32)).astype(np.float32)
    assert same_bits_or_both_zero(got, ref).all()


def test_q4_1_every_scale(oracle_mod):
    """All 16 codes x every finite binary16 scale, each block with a random
    finite binary16 min, against q*d + m in double rounded once (q*d and m are
    multiples of 2^-24 below 2^20, so the double sum is exact)."""
    d = finite_halves()
    m = np.random.default_rng(21).choice(finite_halves(), d.size)
    q = np.tile(np.concatenate([np.arange(16), np.arange(16)]).astype(np.uint8), d.size)
    got = oracle_mod.dequant(Q4_1, layout.pack_q4_1(q, d, m), q.size)
    ref = (q.astype(np.float64) * np.repeat(d.view(np.float16).astype(np.float64), 32)
           + np.repeat(m.view(np.float16).astype(np.float64), 32)).astype(np.float32)
    ok = same_bits_or_both_zero(got, ref) | (np.isinf(got) & (got == ref))
    assert ok.all(), np.flatnonzero(~ok)[:5]


def test_q4_1_nibble_order_and_pair_plane(oracle_mod):
    """Plane 1 holds {d, m} per group: with d = 1 and m = -8 a group decodes
    like Q4_0 with d = 1, and with d = 0 every element is its group's min."""
    codes = bytes(((i & 15) | ((15 - i) << 4)) for i in range(16))
    plane0 = np.frombuffer(codes * 8, np.uint8)
    dm = np.array([0x3C00, 0xC800] * 4 + [0x0000, 0x4500] * 4, np.uint16)  # (1, -8) x 4, (0, 5) x 4
    W = layout.assemble(Q4_1, 256, plane0, dm)
    got = oracle_mod.dequant(Q4_1, W, 256)
    assert list(got[0:16]) == [i - 8 for i in range(16)]
    assert list(got[16:32]) == [(15 - i) - 8 for i in range(16)]
    assert (got[128:256] == 5.0).all()


def test_q1_0_every_scale(oracle_mod):
    """Both codes x every finite binary16 scale (one scale per block of 128):
    the bit b stands for 2b - 1, so the element is +d or -d, compared with
    numpy's binary16 -> float32 conversion (negated for b = 0)."""
    d = finite_halves()
    rng = np.random.default_rng(31)
    b = rng.integers(0, 2, 128 * d.size).astype(np.uint8)
    b[0::128], b[1::128] = 0, 1  # both codes in every block
    got = oracle_mod.dequant(Q1_0, layout.pack_q1_0(b, d), b.size)
    dv = np.repeat(d.view(np.float16).astype(np.float32), 128)
    ref = np.where(b == 1, dv, -dv)
    assert (bits(got) == bits(ref)).all()  # signed zeros included: (-1) * (+0) = -0


def test_q1_0_bit_order_hand_bytes(oracle_mod):
    """Element e is bit (e mod 8) of byte e/8 (least significant first), and
    the scale changes every 128 elements."""
    plane0 = np.zeros(32, np.uint8)
    plane0[0], plane0[1], plane0[16] = 0x01, 0x80, 0xFF
    d = np.array([0x3C00, 0x4000], np.uint16)  # 1.0, 2.0
    got = oracle_mod.dequant(Q1_0, layout.assemble(Q1_0, 256, plane0, d), 256)
    want = -np.ones(256, np.float32)
    want[[0, 15]] = 1.0
    want[128:] = -2.0
    want[128:136] = 2.0
    assert np.array_equal(got, want)


def test_q1_0_sign_quantizer_roundtrip(oracle_mod):
    """Eq. (1) with two symmetric levels: quantizing by sign with d = the
    block's mean |x| (as binary16) decodes to sign(x) * d exactly."""
    rng = np.random.default_rng(32)
    x = rng.standard_normal(128 * 64) * 0.02
    d16 = np.abs(x).reshape(-1, 128).mean(axis=1).astype(np.float16)
    b = (x >= 0).astype(np.uint8)
    got = oracle_mod.dequant(Q1_0, layout.pack_q1_0(b, d16), x.size)
    assert np.array_equal(got, np.sign(x) * np.repeat(d16.astype(np.float32), 128))


# --------------------------------------------------------------------------- hand values

def _block_for(name, f):
    """A minimal tensor (256 elements) whose element 0 carries the fields f."""
    h = lambda v: np.array([v], dtype=np.uint16)
    if name == "q8_0":
        q = np.zeros(256, np.int8)
        q[0] = f["q"]
        return layout.pack_q8_0(q, np.repeat(h(f["d"]), 8)), 0
    if name == "q4_0":
        q = np.zeros(256, np.uint8)
        q[0] = f["q"]
        return layout.pack_q4_0(q, np.repeat(h(f["d"]), 8)), 0
    if name == "q1_0":
        b = np.zeros(256, np.uint8)
        b[0] = f["b"]
        return layout.pack_q1_0(b, np.repeat(h(f["d"]), 2)), 0
    if name == "q4_1":
        q = np.zeros(256, np.uint8)
        q[0] = f["q"]
        return layout.pack_q4_1(q, np.repeat(h(f["d"]), 8), np.repeat(h(f["m"]), 8)), 0
    if name in ("q5_0", "q5_1"):
        q = np.zeros(256, np.uint8)
        q[0] = f["q"]
        if name == "q5_0":
            return layout.pack_q5_0(q, np.repeat(h(f["d"]), 8)), 0
        return layout.pack_q5_1(q, np.repeat(h(f["d"]), 8), np.repeat(h(f["m"]), 8)), 0
    if name == "mxfp4":
        q = np.zeros(256, np.uint8)
        q[0] = f["q"]
        return layout.pack_mxfp4(q, np.full(8, f["E"], np.uint8)), 0
    if name == "q6_k":
        q = np.zeros(256, np.uint8)
        q[0] = f["q"]
        sc = np.zeros(16, np.int8)
        sc[0] = f["sc"]
        return layout.pack_q6_k(q, sc, h(f["d"])), 0
    if name == "q2_k":
        q = np.zeros(256, np.uint8)
        q[0] = f["q"]
        sc = np.zeros(16, np.uint8)
        m = np.zeros(16, np.uint8)
        sc[0], m[0] = f["sc"], f["m"]
        return layout.pack_q2_k(q, sc, m, h(f["d"]), h(f["dmin"])), 0
    q = np.zeros(256, np.uint8)
    q[0] = f["q"]
    sc = np.zeros(8, np.uint8)
    m = np.zeros(8, np.uint8)
    sc[0], m[0] = f["sc"], f["m"]
    if name == "q5_k":
        return layout.pack_q5_k(q, sc, m, h(f["d"]), h(f["dmin"])), 0
    return layout.pack_q4_k(q, sc, m, h(f["d"]), h(f["dmin"])), 0


def test_hand_values(oracle_mod):
    rows = golden_io.hand_values()
    assert len(rows) >= 30
    assert {r[0] for r in rows} >= set(FMT) - {"f16"}
    for name, f, want_bits, want in rows:
        W, e = _block_for(name, f)
        got = oracle_mod.dequant(FMT[name], W, 256)[e]
        assert bits(got) == np.uint32(want_bits), (name, f, hex(int(bits(got))), hex(want_bits))
        assert got == np.float32(want) or (np.isinf(want) and got == np.float32(want))


def test_q4_0_nibble_order_hand_bytes(oracle_mod):
    """Byte i of a group holds element i in bits 0-3 and element i+16 in bits 4-7."""
    codes = bytes(((i & 15) | ((15 - i) << 4)) for i in range(16))  # group 0
    codes += bytes([0x8F] * 16)                                      # group 1
    plane0 = np.frombuffer(codes * 4, np.uint8)                       # 8 groups = 256 elements
    d = np.full(8, 0x3C00, np.uint16)                                 # d = 1
    W = layout.assemble(Q4_0, 256, plane0, d)
    got = oracle_mod.dequant(Q4_0, W, 256)
    assert list(got[0:16]) == [i - 8 for i in range(16)]
    assert list(got[16:32]) == [(15 - i) - 8 for i in range(16)]
    assert list(got[32:48]) == [7.0] * 16          # 0x8F: low nibble 15 -> 7*d
    assert list(got[48:64]) == [0.0] * 16          # high nibble 8 -> 0*d


def test_q4k_scale_record_golden(oracle_mod):
    """The hand-packed record decodes to sc = 1..8, m = 9..16, and the packer
    produces the same bytes."""
    sc, m, rec = golden_io.scale_record()
    assert layout.pack_q4k_records(sc, m).tobytes() == rec
    recs = np.frombuffer(rec * 2, np.uint8)
    # super-block 0: q = 1, d = 1, dmin = 0   -> value = sc_j
    # super-block 1: q = 0, d = 1, dmin = 1   -> value = -m_j
    plane0 = np.concatenate([np.full(128, 0x11, np.uint8), np.zeros(128, np.uint8)])
    dd = np.array([0x3C00, 0x0000, 0x3C00, 0x3C00], np.uint16)
    W = layout.assemble(Q4_K, 512, plane0, recs, dd)
    got = oracle_mod.dequant(Q4_K, W, 512)
    assert list(got[0:256:32]) == [float(v) for v in sc]
    assert all((got[32 * j:32 * j + 32] == sc[j]).all() for j in range(8))
    assert list(got[256::32]) == [-float(v) for v in m]


# --------------------------------------------------------------------------- fuzz: exact reference

def _halves_exact(hb):
    return hb.view(np.float16).astype(np.float64)


def test_q4_k_fuzz_any_finite_scales(oracle_mod):
    """Random fields with scales over all finite binary16 values (subnormals,
    negatives, extremes) against the exact double value rounded once. For every
    finite binary16 d, dmin the double difference is exact, so numpy's
    float64 -> float32 cast is the single correct rounding."""
    rng = np.random.default_rng(1234)
    nsb = 4096
    n = 256 * nsb
    fin = finite_halves()
    q = rng.integers(0, 16, n, dtype=np.uint8)
    sc = rng.integers(0, 64, n // 32, dtype=np.uint8)
    m = rng.integers(0, 64, n // 32, dtype=np.uint8)
    d = rng.choice(fin, nsb)
    dmin = rng.choice(fin, nsb)
    got = oracle_mod.dequant(Q4_K, layout.pack_q4_k(q, sc, m, d, dmin), n)
    D = np.repeat(_halves_exact(d), 256)
    Dm = np.repeat(_halves_exact(dmin), 256)
    SC = np.repeat(sc.astype(np.float64), 32)
    MM = np.repeat(m.astype(np.float64), 32)
    ref = (D * SC * q.astype(np.float64) - Dm * MM).astype(np.float32)
    ok = same_bits_or_both_zero(got, ref) | (np.isinf(got) & (got == ref))
    assert ok.all(), np.flatnonzero(~ok)[:5]


def test_q4_k_fuzz_config_ranges(oracle_mod):
    from paper_2605_20706_amd import synth
    rng = np.random.default_rng(7)
    n = 256 * 1024
    f = synth.gen_fields(Q4_K, n, rng)
    got = oracle_mod.dequant(Q4_K, synth.pack_fields(Q4_K, f), n)
    ref = (np.repeat(f["d"].astype(np.float64), 256) * np.repeat(f["sc"].astype(np.float64), 32)
           * f["q"].astype(np.float64)
           - np.repeat(f["dmin"].astype(np.float64), 256) * np.repeat(f["m"].astype(np.float64), 32))
    assert same_bits_or_both_zero(got, ref.astype(np.float32)).all()


def test_random_bytes_generator_matches_fields_decode(oracle_mod):
    """gen_packed draws the Q4 code plane as random bytes; decoding it element
    by element must give codes in [0, 15] with both nibbles used."""
    from paper_2605_20706_amd import synth
    n = 256 * 64
    W = synth.gen_packed(Q4_0, n, np.random.default_rng(3))
    got = oracle_mod.dequant(Q4_0, W, n)
    offs, _ = layout.plane_offsets(Q4_0, n)
    d = np.repeat(W[offs[1]:offs[1] + 2 * (n // 32)].view(np.float16).astype(np.float64), 32)
    q = got.astype(np.float64) / d + 8
    assert np.array_equal(q, np.round(q)) and q.min() == 0 and q.max() == 15


# --------------------------------------------------------------------------- Eq. (1) round trip

def _round_half_away(v):
    return np.sign(v) * np.floor(np.abs(v) + 0.5)


def test_roundtrip_q8_0_q4_0_eq1(oracle_mod):
    """Quantize per Eq. (1) with an abs-max block scale, dequantize with the
    oracle: every element is within s/2 of the original (clamped codes aside)."""
    rng = np.random.default_rng(11)
    n = 32 * 2048
    w = rng.standard_normal(n) * 0.02
    blocks = w.reshape(-1, 32)
    amax = np.abs(blocks).max(axis=1)
    # q8_0: d = amax / 127, q = round(w / d)
    d8 = (amax / 127).astype(np.float16)
    s8 = np.repeat(d8.astype(np.float64), 32)
    q8 = np.clip(_round_half_away(w / s8), -127, 127)
    got8 = oracle_mod.dequant(Q8_0, layout.pack_q8_0(q8.astype(np.int8), d8), n).astype(np.float64)
    in8 = np.abs(_round_half_away(w / s8)) <= 127
    assert (np.abs(w - got8)[in8] <= s8[in8] / 2 * (1 + 1e-6)).all()
    assert in8.mean() > 0.99
    # q4_0: d = amax / 7, q = round(w / d) + 8 in [0, 15]
    d4 = (amax / 7).astype(np.float16)
    s4 = np.repeat(d4.astype(np.float64), 32)
    raw = _round_half_away(w / s4) + 8
    q4 = np.clip(raw, 0, 15)
    got4 = oracle_mod.dequant(Q4_0, layout.pack_q4_0(q4.astype(np.uint8), d4), n).astype(np.float64)
    in4 = (raw >= 0) & (raw <= 15)
    assert (np.abs(w - got4)[in4] <= s4[in4] / 2 * (1 + 1e-6)).all()
    assert in4.mean() > 0.95


def test_roundtrip_q4_1_eq1(oracle_mod):
    """Eq. (1) with an offset per block: m = the block minimum, d = the block
    range / 15 (both rounded to binary16), q = round((w - m) / d) in [0, 15];
    the oracle's d*q + m is within d/2 of w (plus one float32 rounding)."""
    rng = np.random.default_rng(13)
    n = 32 * 2048
    w = rng.standard_normal(n) * 0.02
    blocks = w.reshape(-1, 32)
    m16 = blocks.min(axis=1).astype(np.float16)
    d16 = ((blocks.max(axis=1) - m16.astype(np.float64)) / 15).astype(np.float16)
    s = np.repeat(d16.astype(np.float64), 32)
    mu = np.repeat(m16.astype(np.float64), 32)
    raw = _round_half_away((w - mu) / s)
    q = np.clip(raw, 0, 15)
    got = oracle_mod.dequant(Q4_1, layout.pack_q4_1(q.astype(np.uint8), d16, m16), n).astype(np.float64)
    inr = (raw >= 0) & (raw <= 15)
    tol = s / 2 + np.abs(got) * 2.0 ** -24
    assert (np.abs(w - got)[inr] <= tol[inr] * (1 + 1e-9)).all()
    assert inr.mean() > 0.95


def test_roundtrip_q4_k_eq1(oracle_mod):
    """K-quant style: x_hat = (d*sc) * q - dmin*m (Eq. (1) with s = d*sc, mu = -dmin*m)."""
    rng = np.random.default_rng(12)
    n = 256 * 512
    from paper_2605_20706_amd import synth
    f = synth.gen_fields(Q4_K, n, rng)
    s = np.repeat(f["d"].astype(np.float64), 256) * np.repeat(f["sc"].astype(np.float64), 32)
    mu = np.repeat(f["dmin"].astype(np.float64), 256) * np.repeat(f["m"].astype(np.float64), 32)
    w = (rng.uniform(-0.5, 15.5, n)) * s - mu
    ok = s > 0
    q = np.zeros(n)
    q[ok] = np.clip(_round_half_away((w[ok] + mu[ok]) / s[ok]), 0, 15)
    got = oracle_mod.dequant(Q4_K, layout.pack_q4_k(q.astype(np.uint8), f["sc"], f["m"], f["d"], f["dmin"]),
                             n).astype(np.float64)
    # one float32 rounding of the result on top of the s/2 bound
    tol = s / 2 + np.abs(got) * 2.0 ** -24
    assert (np.abs(w - got)[ok] <= tol[ok] * (1 + 1e-9)).all()


# --------------------------------------------------------------------------- 5-bit, 6-bit, 2-bit formats

def test_plane_sizes4_golden(oracle_mod):
    for name, n, o1, o2, o3, total in golden_io.plane_sizes4():
        assert oracle_mod.weight_bytes(FMT[name], n) == total, name
        offs, tot = layout.plane_offsets4(FMT[name], n)
        assert (offs[1], offs[2], offs[3], tot) == (o1, o2, o3, total), name


def test_q5_0_exhaustive(oracle_mod):
    """32 codes x every finite binary16 d against the exact products (q - 16) * d."""
    d = finite_halves()
    for q in range(32):
        codes = np.full(d.size * 32, q, np.uint8)
        W = layout.pack_q5_0(codes, d)
        got = oracle_mod.dequant(Q5_0, W, codes.size)[::32]
        ref = (np.float64(q - 16) * d.view(np.float16).astype(np.float64)).astype(np.float32)
        assert same_bits_or_both_zero(got, ref).all(), q


def test_q5_1_every_scale(oracle_mod):
    """Every finite d with random finite mins: q*d + m rounded once (the
    double sum is exact), against numpy's cast of the double sum."""
    d = finite_halves()
    rng = np.random.default_rng(31)
    m = rng.choice(finite_halves(), d.size)
    q = rng.integers(0, 32, d.size).astype(np.uint8)
    codes = np.zeros(d.size * 32, np.uint8)
    codes[::32] = q
    got = oracle_mod.dequant(Q5_1, layout.pack_q5_1(codes, d, m), codes.size)[::32]
    ref = (q.astype(np.float64) * d.view(np.float16).astype(np.float64)
           + m.view(np.float16).astype(np.float64)).astype(np.float32)
    ok = np.isfinite(ref)
    assert same_bits_or_both_zero(got[ok], ref[ok]).all()


@pytest.mark.parametrize("fmt", [Q5_K, Q2_K])
def test_k_quant_fuzz_exact(oracle_mod, fmt):
    """Random d, dmin (any finite binary16), scales, mins and codes: the exact
    d*sc*q - dmin*m (fractions) rounded once."""
    from fractions import Fraction
    rng = np.random.default_rng(32 + fmt)
    n = 256 * 64
    hq = 32 if fmt == Q5_K else 4
    hs = 64 if fmt == Q5_K else 16
    per = 32 if fmt == Q5_K else 16
    q = rng.integers(0, hq, n).astype(np.uint8)
    sc = rng.integers(0, hs, n // per).astype(np.uint8)
    m = rng.integers(0, hs, n // per).astype(np.uint8)
    d = rng.choice(finite_halves(), n // 256)
    dmin = rng.choice(finite_halves(), n // 256)
    W = (layout.pack_q5_k(q, sc, m, d, dmin) if fmt == Q5_K else layout.pack_q2_k(q, sc, m, d, dmin))
    got = oracle_mod.dequant(fmt, W, n)
    dd = d.view(np.float16).astype(np.float64)
    dm = dmin.view(np.float16).astype(np.float64)
    for e in rng.integers(0, n, 3000):
        S, j = e // 256, e // per
        v = Fraction(dd[S]) * int(sc[j]) * int(q[e]) - Fraction(dm[S]) * int(m[j])
        assert got[e] == np.float32(float(v)) or (got[e] == 0 and v == 0), (e, float(v), got[e])
        # the nearest float of the exact value: within half an ulp
        assert abs(Fraction(float(got[e])) - v) <= Fraction(float(np.spacing(np.float32(abs(float(v)))))) / 2


def test_q6_k_codes_and_scales_exhaustive(oracle_mod):
    """Every 6-bit code x every int8 scale for three binary16 d (one a
    subnormal), and every finite d for one code and scale: d*sc*(q - 32) is
    exact in float32 (<= 23 significant bits)."""
    for dbits in (0x3C00, 0x2E66, 0x0003):
        q = np.tile(np.arange(64, dtype=np.uint8), 256 * 16)           # element e: code e mod 64
        sc = np.repeat(np.arange(-128, 128, dtype=np.int16), 4).astype(np.int8)  # 16 elements per scale
        n = q.size
        sc = np.resize(sc, n // 16)
        W = layout.pack_q6_k(q, sc, np.full(n // 256, dbits, np.uint16))
        got = oracle_mod.dequant(Q6_K, W, n)
        dv = np.array([dbits], np.uint16).view(np.float16).astype(np.float64)[0]
        ref = (dv * np.repeat(sc.astype(np.float64), 16) * (q.astype(np.float64) - 32)).astype(np.float32)
        assert same_bits_or_both_zero(got, ref).all(), dbits
    d = finite_halves()
    q = np.zeros(d.size * 256, np.uint8)
    q[::256] = 63
    sc = np.zeros(d.size * 16, np.int8)
    sc[::16] = -77
    got = oracle_mod.dequant(Q6_K, layout.pack_q6_k(q, sc, d), q.size)[::256]
    ref = (d.view(np.float16).astype(np.float64) * -77 * 31).astype(np.float32)
    ok = np.isfinite(ref)
    assert same_bits_or_both_zero(got[ok], ref[ok]).all()


def test_high_bit_planes_hand_bytes(oracle_mod):
    """Fifth bits (q5): element e at bit e mod 8 of byte e/8 of plane 1;
    high two bits (q6_k) and 2-bit codes (q2_k): element e at bits 2(e mod 4)
    of byte e/4; q2_k scale in bits 0-3, min in bits 4-7 of a sub-block's byte."""
    n = 256
    # q5_0: low nibbles all 0, fifth bits 0b00000101 in byte 0 -> elements 0 and 2 have q = 16
    plane0 = np.zeros(n // 2, np.uint8)
    plane1 = np.zeros(n // 8, np.uint8)
    plane1[0] = 0x05
    W = layout.assemble(Q5_0, n, plane0, plane1, np.full(n // 32, 0x3C00, np.uint16))
    got = oracle_mod.dequant(Q5_0, W, n)
    assert list(got[:4]) == [0.0, -16.0, 0.0, -16.0]
    # q6_k: nibbles 0, high-bit byte 0 = 0b11100100 -> elements 0..3 have high bits 0, 1, 2, 3
    p0 = np.zeros(n // 2, np.uint8)
    p1 = np.zeros(n // 4, np.uint8)
    p1[0] = 0b11100100
    p2 = np.ones(n // 16, np.int8)
    W = layout.assemble(Q6_K, n, p0, p1, p2, np.array([0x3C00], np.uint16))
    got = oracle_mod.dequant(Q6_K, W, n)
    assert list(got[:5]) == [-32.0, -16.0, 0.0, 16.0, -32.0]
    # q2_k: code byte 0 = 0b00011011 -> elements 0..3 codes 3, 2, 1, 0; sub-block 0's byte = 0x21
    #   (scale 1, min 2); d = 1, dmin = 0.5 -> values q - 1
    c = np.zeros(n // 4, np.uint8)
    c[0] = 0b00011011
    scm = np.zeros(n // 16, np.uint8)
    scm[0] = 0x21
    dd = np.array([0x3C00, 0x3800], np.uint16)
    W = layout.assemble(Q2_K, n, c, scm, dd)
    got = oracle_mod.dequant(Q2_K, W, n)
    assert list(got[:5]) == [2.0, 1.0, 0.0, -1.0, -1.0]
    assert list(got[16:18]) == [0.0, 0.0]   # sub-block 1: scale 0, min 0


@pytest.mark.parametrize("fmt", [Q5_0, Q5_1, Q5_K, Q6_K, Q2_K])
def test_roundtrip_eq1_new_formats(oracle_mod, fmt):
    """Weights from N(0, 0.02^2) encoded by the Eq. (1) test quantizer:
    every element whose code was not clamped is within s/2 of the original
    (s the element's effective scale), plus one float32 rounding."""
    from paper_2605_20706_amd import synth
    rng = np.random.default_rng(40 + fmt)
    n = 256 * 256
    f = synth.gen_fields_eq1(fmt, n, np.random.default_rng(40 + fmt))
    w = np.random.default_rng(40 + fmt).standard_normal(n) * 0.02   # the same draw
    got = oracle_mod.dequant(fmt, synth.pack_fields(fmt, f), n).astype(np.float64)
    if fmt in (Q5_0, Q5_1):
        s = np.repeat(f["d"].astype(np.float64), 32)
    elif fmt == Q5_K:
        s = np.repeat(f["d"].astype(np.float64), 256) * np.repeat(f["sc"].astype(np.float64), 32)
    else:
        s = np.abs(np.repeat(f["d"].astype(np.float64), 256) * np.repeat(f["sc"].astype(np.float64), 16))
    top = {Q5_0: 31, Q5_1: 31, Q5_K: 31, Q6_K: 63, Q2_K: 3}[fmt]
    inner = (f["q"] > 0) & (f["q"] < top) & (s > 0)
    tol = s / 2 + np.abs(got) * 2.0 ** -24
    assert (np.abs(w - got)[inner] <= tol[inner] * (1 + 1e-9)).all()
    assert inner.mean() > 0.5
    del rng


# --------------------------------------------------------------------------- mxfp4

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def test_mxfp4_every_code_every_exponent(oracle_mod):
    """16 codes x all 256 e8m0 exponents against numpy: the e2m1 magnitude
    table (from its definition, by hand) times 2^(E - 127) with numpy's
    ldexp, cast to float32 (overflow to +-inf); E = 255 is NaN."""
    E = np.repeat(np.arange(256), 1).astype(np.uint8)
    codes = np.tile(np.concatenate([np.arange(16), np.arange(16)]).astype(np.uint8), E.size)
    got = oracle_mod.dequant(MXFP4, layout.pack_mxfp4(codes, E), codes.size).reshape(256, 32)
    mag = E2M1[np.arange(16) & 7] * np.where(np.arange(16) >= 8, -1.0, 1.0)
    with np.errstate(over="ignore"):
        ref = (np.ldexp(np.tile(mag, 2)[None, :], (np.arange(256) - 127)[:, None])).astype(np.float32)
    nan = np.arange(256) == 255
    assert np.isnan(got[nan]).all()
    assert same_bits_or_both_zero(got[~nan], ref[~nan]).all()
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))  # -0 for code 8


def test_mxfp4_roundtrip_eq1(oracle_mod):
    """Gaussian weights encoded with the largest magnitude at or below
    6 * 2^(E - 127) and each weight at its nearest e2m1 level: the error is
    at most half the local level spacing (0.25, 0.5 or 1 times the scale)."""
    from paper_2605_20706_amd import synth
    n = 32 * 4096
    f = synth.gen_fields_eq1(MXFP4, n, np.random.default_rng(44))
    w = np.random.default_rng(44).standard_normal(n) * 0.02
    got = oracle_mod.dequant(MXFP4, synth.pack_fields(MXFP4, f), n).astype(np.float64)
    s = np.repeat(np.ldexp(1.0, f["E"].astype(np.int64) - 127), 32)
    a = np.abs(w) / s
    half_gap = np.where(a <= 2, 0.25, np.where(a <= 4, 0.5, 1.0))
    assert (np.abs(w - got) <= half_gap * s * (1 + 1e-12)).all()
    assert (np.abs(w) <= 6 * s).all()
