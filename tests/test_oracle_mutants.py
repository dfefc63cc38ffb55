"""The oracle's pins catch planted mistakes.

Each case copies oracle/lw_oracle.c, plants one plausible mistake in the copy
(a dropped term, a wrong sign or offset, a swapped or transposed operand, a
wrong bit position, a double rounding, a misplaced plane), builds it with the
oracle's own flags and runs the pin modules against it (LW_ORACLE_LIB points
the oracle package at the copy). Every mutant must make at least one pin
fail; the unmodified copy must pass them all. Nothing here touches the GPU or
the HIP library."""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "lw_oracle.c")
PINS = ["tests/test_oracle_formats.py", "tests/test_oracle_gemv.py", "tests/test_oracle_termmass.py",
        "tests/test_oracle_attn.py"]

# (name, text in the oracle, replacement); every occurrence is replaced.
MUTANTS = [
    ("q4_0 offset -7 instead of -8", "return (double)(q - 8) * d;", "return (double)(q - 7) * d;"),
    ("q4_k min term dropped", "return a - b;", "return a;"),
    ("q4_k min term added", "return a - b;", "return a + b;"),
    ("q4_k d*sc rounded to binary16 precision", "double a = d * (double)sc * (double)q;",
     "double a = ldexp(rint(ldexp(d * (double)sc, 10 - ilogb(d * (double)sc))), ilogb(d * (double)sc) - 10)"
     " * (double)q;"),
    ("q4_k value rounded toward zero", "return a - b;", "return (double)nextafterf((float)(a - b), 0.0f);"),
    ("q4 nibbles swapped", "return i < 16 ? (byte & 15u) : (byte >> 4);",
     "return i < 16 ? (byte >> 4) : (byte & 15u);"),
    ("q8_0 codes unsigned", "int q = (int)(int8_t)W[e];", "int q = (int)W[e];"),
    ("binary16 exponent bias off by one", "ldexp((double)(1024u + f), (int)e - 25)",
     "ldexp((double)(1024u + f), (int)e - 24)"),
    ("binary16 subnormals halved", "v = ldexp((double)f, -24);", "v = ldexp((double)f, -25);"),
    ("q4_k min field at the wrong bit", "bit_field(rec, 48 + 6 * j, 6)", "bit_field(rec, 42 + 6 * j, 6)"),
    ("q4_k scale and min fields swapped", "unsigned sc = bit_field(rec, 6 * j, 6);",
     "unsigned sc = bit_field(rec, 48 + 6 * j, 6);"),
    ("q4_1 min subtracted", "return (double)q * d + m;", "return (double)q * d - m;"),
    ("q1_0 level 2b instead of 2b - 1", "return (double)(2 * b - 1) * d;", "return (double)(2 * b) * d;"),
    ("q1_0 bits read most-significant first", "(W[e / 8] >> (e % 8)) & 1", "(W[e / 8] >> (7 - e % 8)) & 1"),
    ("x operand transposed", "double p = (double)w[k] * (double)xt[k];",
     "double p = (double)w[k] * (double)xt[jb->K - 1 - k];"),
    ("last product dropped", "            for (int64_t k = 0; k < jb->K; ++k) {\n                double p",
     "            for (int64_t k = 0; k + 1 < jb->K; ++k) {\n                double p"),
    ("condition sum without magnitudes", "a += fabs(p);", "a += p;"),
    ("scale plane not aligned", "off[1] = round_up_256(n / 2);", "off[1] = n / 2;"),
    ("legacy scale of the even group used for the odd one", "W + off[1] + 2 * (e / 32)",
     "W + off[1] + 2 * ((e / 32) / 2 * 2)"),
    ("q5 fifth bit ignored", "return q4_code(W, e) | (hi << 4);", "return q4_code(W, e);"),
    ("q5_0 offset -15", "return (double)(q - 16) * d;", "return (double)(q - 15) * d;"),
    ("q6_k high bits at the wrong place", "return q4_code(W, e) | (two_bits(W + off[1], e) << 4);",
     "return q4_code(W, e) | (two_bits(W + off[1], e) << 3);"),
    ("q6_k scales read unsigned", "int sc = (int)(int8_t)W[off[2] + e / 16];", "int sc = (int)W[off[2] + e / 16];"),
    ("q6_k scale per 32 instead of 16", "int sc = (int)(int8_t)W[off[2] + e / 16];",
     "int sc = (int)(int8_t)W[off[2] + e / 32];"),
    ("q2_k scale and min nibbles swapped", "unsigned sc = scm & 15u, m = scm >> 4;",
     "unsigned sc = scm >> 4, m = scm & 15u;"),
    ("2-bit fields read most-significant first", "return bit_field(plane + e / 4, 2 * (int)(e % 4), 2);",
     "return bit_field(plane + e / 4, 6 - 2 * (int)(e % 4), 2);"),
    ("attention: key/value head of a query head taken modulo", "int64_t g = h / group;", "int64_t g = h % n_kv_heads;"),
    ("attention: scale dropped", "s[j] = scale * acc;", "s[j] = acc;"),
    ("attention: values read from the key cache",
     "double v = (double)(float)exact_value(fmt, Vc, offv, (g * kv_len + j) * head_dim + d);",
     "double v = (double)(float)exact_value(fmt, Kc, offv, (g * kv_len + j) * head_dim + d);"),
    ("attention: last position skipped in the normalisation", "        for (int64_t j = 0; j < kv_len; ++j) {\n            s[j] = exp(s[j] - smax);",
     "        for (int64_t j = 0; j + 1 < kv_len; ++j) {\n            s[j] = exp(s[j] - smax);"),
    ("e2m1 exponent bias 0", "return ldexp(1.0 + 0.5 * (double)m, (int)e - 1);",
     "return ldexp(1.0 + 0.5 * (double)m, (int)e);"),
    ("e2m1 sign ignored", "return (c & 8u) ? -v : v;", "return v;"),
    ("e8m0 bias 126", "double v = e2m1_magnitude(c) * ldexp(1.0, (int)E - 127);",
     "double v = e2m1_magnitude(c) * ldexp(1.0, (int)E - 126);"),
    ("term mass without the code shift", "return fabs(s) * (q + (double)beta) + fabs(mu - (double)beta * s);",
     "return fabs(s) * q + fabs(mu - (double)beta * s);"),
    ("term mass offset taken with its sign", "fabs(mu - (double)beta * s);", "(mu - (double)beta * s);"),
]


def build(dirpath, text):
    src = os.path.join(dirpath, "lw_oracle.c")
    lib = os.path.join(dirpath, "liboracle.so")
    with open(src, "w") as fh:
        fh.write(text)
    subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                           "-pthread", "-o", lib, src, "-lm"])
    return lib


def run_pins(lib):
    env = dict(os.environ, LW_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"]
                       + PINS, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, (r.stdout + r.stderr)[-600:]


@pytest.fixture(scope="module")
def original():
    with open(SRC) as fh:
        return fh.read()


def test_unmodified_copy_passes(original):
    with tempfile.TemporaryDirectory() as d:
        rc, out = run_pins(build(d, original))
    assert rc == 0, out


def test_every_planted_mistake_is_caught(original):
    for name, old, new in MUTANTS:
        assert old in original, "mutation anchor missing: %s" % name

    def one(case):
        name, old, new = case
        with tempfile.TemporaryDirectory() as d:
            rc, out = run_pins(build(d, original.replace(old, new)))
        return name, rc, out

    with ThreadPoolExecutor(4) as ex:
        results = list(ex.map(one, MUTANTS))
    missed = [(name, out) for name, rc, out in results if rc == 0]
    assert not missed, "planted mistakes no pin caught: %s" % [m[0] for m in missed]
    # a mutant must fail a pin, not the collection or the build
    broken = [(name, out) for name, rc, out in results if rc not in (0, 1)]
    assert not broken, broken
