"""Seeded synthetic inputs with the shapes and value distributions of the
decode workloads (Llama-3.2-1B- and Llama-3-8B-shaped weight sets).

Draws fields with numpy's PCG64 generator and lays them out with ``layout``;
holds none of the method's arithmetic (no dequantization, no product). Both
the HIP library's tests and the CPU oracle read the bytes produced here.

Recipe (each matrix has its own generator,
``default_rng(SeedSequence([0, workload_id, layer, matrix_id]))``; the single
Q8_0 matrix uses the literal seed 0):

* f16   w ~ N(0, 0.02^2) drawn as float32 and rounded to binary16 (RNE);
* q8_0  codes uniform in [-127, 127]; d uniform in [1e-3, 2e-2] -> binary16;
* q4_0  codes uniform in [0, 15] (drawn as uniform random bytes, i.e. two
        independent uniform nibbles per byte); d uniform in [1e-3, 2e-2];
* q4_k  codes as q4_0; sc and m uniform in [0, 63]; d and dmin uniform in
        [1e-4, 2e-3] -> binary16;
* q4_1  codes as q4_0; d uniform in [1e-3, 2e-2] and m uniform in [-0.2, 0]
        -> binary16 (a block's values span [m, m + 15 d], as for weights
        quantized against their block minimum);
* q1_0  bits uniform in {0, 1} (uniform random bytes); d uniform in
        [1e-3, 2e-2] -> binary16 (one per 128 weights);
* q5_0  codes uniform in [0, 31]; d as q4_0;   q5_1  codes as q5_0, d and m as q4_1;
* q5_k  codes as q5_0; sc, m, d, dmin as q4_k;
* q6_k  codes uniform in [0, 63]; int8 scales uniform in [-128, 127]; d uniform in
        [1e-5, 2e-4] -> binary16 (the lower part binary16 subnormals);
* q2_k  codes uniform in [0, 3]; 4-bit scales and mins uniform in [0, 15]; d and
        dmin as q4_k;
* mxfp4 e2m1 codes uniform in [0, 15]; e8m0 exponents uniform in [118, 124]
        (block scales 2^-9 .. 2^-3, weights up to 6 * 2^-3);
* x     float32 N(0, 1), shape [n_tok, K], from the generator of the workload
        (matrix_id 99).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import layout
from .layout import F16, MXFP4, Q1_0, Q2_K, Q4_0, Q4_1, Q4_K, Q5_0, Q5_1, Q5_K, Q6_K, Q8_0


@dataclass(frozen=True)
class Matrix:
    name: str
    M: int
    K: int
    layer: int
    matrix_id: int


@dataclass(frozen=True)
class Workload:
    key: str
    workload_id: int
    fmt: int
    matrices: tuple
    n_toks: tuple = (1,)
    description: str = ""

    @property
    def weights(self) -> int:
        return sum(m.M * m.K for m in self.matrices)


def _llama_layers(n_layers, hidden, qkv, ffn):
    mats = []
    for L in range(n_layers):
        mats += [Matrix("qkv", qkv, hidden, L, 0), Matrix("o", hidden, hidden, L, 1),
                 Matrix("gate", ffn, hidden, L, 2), Matrix("up", ffn, hidden, L, 3),
                 Matrix("down", hidden, ffn, L, 4)]
    return mats


# Llama-3.2-1B: hidden 2048, 32 q-heads / 8 kv-heads of 64 -> QKV 3072, FFN 8192, 16 layers.
_L1B = dict(n_layers=16, hidden=2048, qkv=3072, ffn=8192)
# Llama-3-8B: hidden 4096, kv width 1024 -> QKV 6144, FFN 14336, 32 layers.
_L8B = dict(n_layers=32, hidden=4096, qkv=6144, ffn=14336)
_VOCAB = 128256
# A 1.7B-parameter decoder for the 1-bit format: hidden 2048, 16 q-heads / 8
# kv-heads of 128 -> QKV 4096, FFN 6144, 28 layers, vocabulary 151936
# (1.72e9 weights; at 1.125 bits per weight 0.24 GB).
_L1B7 = dict(n_layers=28, hidden=2048, qkv=4096, ffn=6144)
_VOCAB_1B7 = 151936

WORKLOADS = {
    "q8_0_2048": Workload("q8_0_2048", 1, Q8_0, (Matrix("w", 2048, 2048, 0, 0),),
                          description="single Q8_0 GEMV 2048x2048, 1 token"),
    "f16_llama1b": Workload("f16_llama1b", 2, F16, tuple(_llama_layers(**_L1B)),
                            description="f16 GEMV over the 80 per-layer decode matrices of a "
                                        "Llama-3.2-1B-shaped model, 1 token"),
    "q4_0_llama1b": Workload("q4_0_llama1b", 3, Q4_0,
                             tuple(_llama_layers(**_L1B)) + (Matrix("lm_head", _VOCAB, 2048, 16, 5),),
                             description="Q4_0 decode-step weight set, Llama-3.2-1B shapes + lm_head, "
                                         "1 token"),
    "q4_k_llama8b": Workload("q4_k_llama8b", 4, Q4_K,
                             tuple(_llama_layers(**_L8B)) + (Matrix("lm_head", _VOCAB, 4096, 32, 5),),
                             description="Q4_K-style decode-step weight set, Llama-3-8B shapes "
                                         "(32 layers) + lm_head, 1 token"),
    "q4_0_llama8b_ffn": Workload("q4_0_llama8b_ffn", 5, Q4_0,
                                 (Matrix("gate", 14336, 4096, 0, 2), Matrix("up", 14336, 4096, 0, 3),
                                  Matrix("down", 4096, 14336, 0, 4)),
                                 n_toks=(1, 2, 4, 8, 512),
                                 description="multi-token Q4_0 on Llama-3-8B gate/up/down, "
                                             "n_tok in {1,2,4,8} and prefill 512"),
    "q4_1_llama8b_ffn": Workload("q4_1_llama8b_ffn", 6, Q4_1,
                                 (Matrix("gate", 14336, 4096, 0, 2), Matrix("up", 14336, 4096, 0, 3),
                                  Matrix("down", 4096, 14336, 0, 4)),
                                 n_toks=(1, 2, 4, 8, 512),
                                 description="Q4_1 (blocks with a min) on Llama-3-8B gate/up/down, "
                                             "n_tok in {1,2,4,8} and prefill 512"),
    **{"%s_llama8b_ffn" % name: Workload("%s_llama8b_ffn" % name, wid, fmt,
                                        (Matrix("gate", 14336, 4096, 0, 2), Matrix("up", 14336, 4096, 0, 3),
                                         Matrix("down", 4096, 14336, 0, 4)),
                                        n_toks=(1, 2, 4, 8, 512),
                                        description="%s on Llama-3-8B gate/up/down, n_tok in {1,2,4,8} and "
                                                    "prefill 512" % desc)
       for name, wid, fmt, desc in (("q5_0", 8, Q5_0, "Q5_0 (5-bit legacy blocks)"),
                                    ("q5_1", 9, Q5_1, "Q5_1 (5-bit legacy blocks with a min)"),
                                    ("q5_k", 10, Q5_K, "Q5_K-style (5-bit K-quant)"),
                                    ("q6_k", 11, Q6_K, "Q6_K-style (6-bit K-quant, 16-element sub-blocks)"),
                                    ("q2_k", 12, Q2_K, "Q2_K-style (2-bit K-quant, 16-element sub-blocks)"),
                                    ("mxfp4", 13, MXFP4, "mxfp4 (e2m1 with an e8m0 scale per 32)"))},
    "q1_0_1b7": Workload("q1_0_1b7", 7, Q1_0,
                         tuple(_llama_layers(**_L1B7)) + (Matrix("lm_head", _VOCAB_1B7, 2048, 28, 5),),
                         description="q1_0 (1 bit, one scale per 128) decode-step weight set of a "
                                     "1.7B-parameter decoder (28 layers) + lm_head, 1 token"),
}


def rng_for(workload_id: int, layer: int, matrix_id: int) -> np.random.Generator:
    if workload_id == 1:
        return np.random.default_rng(0)
    return np.random.default_rng(np.random.SeedSequence([0, workload_id, layer, matrix_id]))


def _uniform_half(rng, lo, hi, size):
    return rng.uniform(lo, hi, size).astype(np.float16)


def _random_bytes(rng, nbytes):
    """Uniform random bytes: little-endian bytes of uniform 64-bit draws."""
    words = (nbytes + 7) // 8
    return rng.integers(0, 2 ** 64 - 1, words, dtype=np.uint64, endpoint=True).view(np.uint8)[:nbytes]


def gen_fields(fmt: int, n: int, rng: np.random.Generator) -> dict:
    """Fields of n elements drawn per the recipe (4-bit codes as explicit
    values in [0, 15]; meant for sizes where an array of n bytes is cheap)."""
    if fmt == F16:
        return {"w": (rng.standard_normal(n, dtype=np.float32) * np.float32(0.02)).astype(np.float16)}
    if fmt == Q8_0:
        return {"q": rng.integers(-127, 128, n, dtype=np.int8),
                "d": _uniform_half(rng, 1e-3, 2e-2, n // 32)}
    if fmt == Q4_0:
        return {"q": rng.integers(0, 16, n, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-3, 2e-2, n // 32)}
    if fmt == Q4_1:
        return {"q": rng.integers(0, 16, n, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-3, 2e-2, n // 32),
                "m": _uniform_half(rng, -0.2, 0.0, n // 32)}
    if fmt == Q1_0:
        return {"b": rng.integers(0, 2, n, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-3, 2e-2, n // 128)}
    if fmt in (Q4_K, Q5_K):
        return {"q": rng.integers(0, 16 if fmt == Q4_K else 32, n, dtype=np.uint8),
                "sc": rng.integers(0, 64, n // 32, dtype=np.uint8),
                "m": rng.integers(0, 64, n // 32, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-4, 2e-3, n // 256),
                "dmin": _uniform_half(rng, 1e-4, 2e-3, n // 256)}
    if fmt == Q5_0:
        return {"q": rng.integers(0, 32, n, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-3, 2e-2, n // 32)}
    if fmt == Q5_1:
        return {"q": rng.integers(0, 32, n, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-3, 2e-2, n // 32),
                "m": _uniform_half(rng, -0.2, 0.0, n // 32)}
    if fmt == Q6_K:
        return {"q": rng.integers(0, 64, n, dtype=np.uint8),
                "sc": rng.integers(-128, 128, n // 16, dtype=np.int8),
                "d": _uniform_half(rng, 1e-5, 2e-4, n // 256)}
    if fmt == MXFP4:
        return {"q": rng.integers(0, 16, n, dtype=np.uint8),
                "E": rng.integers(118, 125, n // 32, dtype=np.uint8)}
    if fmt == Q2_K:
        return {"q": rng.integers(0, 4, n, dtype=np.uint8),
                "sc": rng.integers(0, 16, n // 16, dtype=np.uint8),
                "m": rng.integers(0, 16, n // 16, dtype=np.uint8),
                "d": _uniform_half(rng, 1e-4, 2e-3, n // 256),
                "dmin": _uniform_half(rng, 1e-4, 2e-3, n // 256)}
    raise ValueError(fmt)


def pack_fields(fmt: int, f: dict) -> np.ndarray:
    if fmt == F16:
        return layout.pack_f16(f["w"])
    if fmt == Q8_0:
        return layout.pack_q8_0(f["q"], f["d"])
    if fmt == Q4_0:
        return layout.pack_q4_0(f["q"], f["d"])
    if fmt == Q4_1:
        return layout.pack_q4_1(f["q"], f["d"], f["m"])
    if fmt == Q1_0:
        return layout.pack_q1_0(f["b"], f["d"])
    if fmt == Q5_0:
        return layout.pack_q5_0(f["q"], f["d"])
    if fmt == Q5_1:
        return layout.pack_q5_1(f["q"], f["d"], f["m"])
    if fmt == Q5_K:
        return layout.pack_q5_k(f["q"], f["sc"], f["m"], f["d"], f["dmin"])
    if fmt == Q6_K:
        return layout.pack_q6_k(f["q"], f["sc"], f["d"])
    if fmt == Q2_K:
        return layout.pack_q2_k(f["q"], f["sc"], f["m"], f["d"], f["dmin"])
    if fmt == MXFP4:
        return layout.pack_mxfp4(f["q"], f["E"])
    return layout.pack_q4_k(f["q"], f["sc"], f["m"], f["d"], f["dmin"])


def gen_packed(fmt: int, n: int, rng: np.random.Generator) -> np.ndarray:
    """n packed elements per the recipe. The 4-bit code plane is drawn as
    uniform random bytes (same distribution as two uniform nibbles)."""
    if fmt in (F16, Q8_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4):
        return pack_fields(fmt, gen_fields(fmt, n, rng))
    offs, total = layout.plane_offsets(fmt, n)
    out = np.zeros(total, dtype=np.uint8)
    if fmt == Q1_0:
        out[0:n // 8] = _random_bytes(rng, n // 8)
        out[offs[1]:offs[1] + 2 * (n // 128)] = _uniform_half(rng, 1e-3, 2e-2, n // 128).view(np.uint8)
        return out
    out[0:n // 2] = _random_bytes(rng, n // 2)
    if fmt == Q4_0:
        out[offs[1]:offs[1] + 2 * (n // 32)] = _uniform_half(rng, 1e-3, 2e-2, n // 32).view(np.uint8)
        return out
    if fmt == Q4_1:
        dm = np.empty((n // 32, 2), dtype=np.float16)
        dm[:, 0] = _uniform_half(rng, 1e-3, 2e-2, n // 32)
        dm[:, 1] = _uniform_half(rng, -0.2, 0.0, n // 32)
        out[offs[1]:offs[1] + 4 * (n // 32)] = dm.view(np.uint8).reshape(-1)
        return out
    sc = rng.integers(0, 64, n // 32, dtype=np.uint8)
    m = rng.integers(0, 64, n // 32, dtype=np.uint8)
    out[offs[1]:offs[1] + 12 * (n // 256)] = layout.pack_q4k_records(sc, m).reshape(-1)
    dd = np.empty((n // 256, 2), dtype=np.float16)
    dd[:, 0] = _uniform_half(rng, 1e-4, 2e-3, n // 256)
    dd[:, 1] = _uniform_half(rng, 1e-4, 2e-3, n // 256)
    out[offs[2]:offs[2] + 4 * (n // 256)] = dd.view(np.uint8).reshape(-1)
    return out


def gen_matrix(wl: Workload, mat: Matrix) -> np.ndarray:
    return gen_packed(wl.fmt, mat.M * mat.K, rng_for(wl.workload_id, mat.layer, mat.matrix_id))


def gen_x(wl: Workload, K: int, n_tok: int = 1) -> np.ndarray:
    rng = rng_for(wl.workload_id, 0, 99) if wl.workload_id != 1 else np.random.default_rng([0, 99])
    return rng.standard_normal((n_tok, K), dtype=np.float32)


def gen_x_seeded(seed, K: int, n_tok: int = 1) -> np.ndarray:
    return np.random.default_rng(seed).standard_normal((n_tok, K), dtype=np.float32)


def algorithmic_bytes(fmt: int, M: int, K: int, n_tok: int = 1) -> float:
    """Bytes the product must move once: packed W + x + y."""
    return layout.BYTES_PER_WEIGHT[fmt] * M * K + 4.0 * n_tok * (K + M)


# ---------------------------------------------------------------------------
# Edge-case inputs for the parity tests. These draw and encode fields only;
# they compute no dequantized value and no product.

def _round_half_away(v):
    return np.sign(v) * np.floor(np.abs(v) + 0.5)


def gen_fields_eq1(fmt: int, n: int, rng: np.random.Generator, sigma: float = 0.02) -> dict:
    """Fields of n weights w ~ N(0, sigma^2) encoded by a test-only Eq. (1)
    quantizer (round half away from zero): the codes then peak at the code of
    zero, as for real weights, instead of being uniform.

    q8_0  d = fp16(amax / 127), q = clamp(round(w / d), -127, 127)
    q4_0  d = fp16(amax / 7), q = clamp(round(w / d) + 8, 0, 15)
    q4_1  m = fp16(min), d = fp16((max - m) / 15), q = clamp(round((w - m) / d), 0, 15)
    q4_k  per sub-block of 32: scale (max - min') / 15 and offset -min' with
          min' = min(min, 0); super-block d, dmin = fp16(largest / 63);
          sc, m = clamp(round(. / d), 0, 63); q = clamp(round((w + dmin m) / (d sc)), 0, 15)
    q1_0  d = fp16(mean |w|) per 128, b = (w >= 0)
    f16   w rounded to binary16
    """
    w = rng.standard_normal(n) * sigma
    if fmt == F16:
        return {"w": w.astype(np.float16)}
    if fmt == Q1_0:
        blk = w.reshape(-1, 128)
        return {"b": (w >= 0).astype(np.uint8), "d": np.abs(blk).mean(axis=1).astype(np.float16)}
    blk = w.reshape(-1, 32)
    if fmt in (Q8_0, Q4_0):
        lim = 127 if fmt == Q8_0 else 7
        d = (np.abs(blk).max(axis=1) / lim).astype(np.float16)
        s = np.repeat(d.astype(np.float64), 32)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away(w / s), 0.0)
        if fmt == Q8_0:
            return {"q": np.clip(r, -127, 127).astype(np.int8), "d": d}
        return {"q": np.clip(r + 8, 0, 15).astype(np.uint8), "d": d}
    if fmt == Q4_1:
        m = blk.min(axis=1).astype(np.float16)
        d = ((blk.max(axis=1) - m.astype(np.float64)) / 15).astype(np.float16)
        s = np.repeat(d.astype(np.float64), 32)
        mu = np.repeat(m.astype(np.float64), 32)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away((w - mu) / s), 0.0)
        return {"q": np.clip(r, 0, 15).astype(np.uint8), "d": d, "m": m}
    if fmt == Q5_0:
        d = (np.abs(blk).max(axis=1) / 15).astype(np.float16)
        s = np.repeat(d.astype(np.float64), 32)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away(w / s), 0.0)
        return {"q": np.clip(r + 16, 0, 31).astype(np.uint8), "d": d}
    if fmt == Q5_1:
        m = blk.min(axis=1).astype(np.float16)
        d = ((blk.max(axis=1) - m.astype(np.float64)) / 31).astype(np.float16)
        s = np.repeat(d.astype(np.float64), 32)
        mu = np.repeat(m.astype(np.float64), 32)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away((w - mu) / s), 0.0)
        return {"q": np.clip(r, 0, 31).astype(np.uint8), "d": d, "m": m}
    if fmt == MXFP4:
        # the block exponent puts the largest magnitude at or below 6 * 2^(E - 127)
        # (E = ceil(log2(amax / 6)) + 127), each weight the nearest e2m1 magnitude
        amax = np.abs(blk).max(axis=1)
        with np.errstate(divide="ignore"):
            E = np.clip(np.ceil(np.log2(np.where(amax > 0, amax, 1.0) / 6.0)) + 127, 0, 254).astype(np.int64)
        s = np.repeat(np.ldexp(1.0, E - 127), 32)
        mags = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
        a = np.abs(w) / s
        idx = np.abs(a[:, None] - mags[None, :]).argmin(axis=1)
        return {"q": (idx + 8 * (w < 0)).astype(np.uint8), "E": E.astype(np.uint8)}
    if fmt == Q6_K:
        b16 = w.reshape(-1, 16)
        scale = np.abs(b16).max(axis=1) / 31
        d = (scale.reshape(-1, 16).max(axis=1) / 127).astype(np.float16)
        dd = np.repeat(d.astype(np.float64), 16)
        with np.errstate(divide="ignore", invalid="ignore"):
            sc = np.clip(np.where(dd > 0, _round_half_away(scale / dd), 0), -128, 127)
        s = np.repeat(dd * sc, 16)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away(w / s), 0.0)
        return {"q": np.clip(r + 32, 0, 63).astype(np.uint8), "sc": sc.astype(np.int8), "d": d}
    if fmt == Q2_K:
        b16 = w.reshape(-1, 16)
        mn = np.minimum(b16.min(axis=1), 0.0)
        scale = (b16.max(axis=1) - mn) / 3
        off = -mn
        d = (scale.reshape(-1, 16).max(axis=1) / 15).astype(np.float16)
        dmin = (off.reshape(-1, 16).max(axis=1) / 15).astype(np.float16)
        dd = np.repeat(d.astype(np.float64), 16)
        dm = np.repeat(dmin.astype(np.float64), 16)
        with np.errstate(divide="ignore", invalid="ignore"):
            sc = np.clip(np.where(dd > 0, _round_half_away(scale / dd), 0), 0, 15)
            mm = np.clip(np.where(dm > 0, _round_half_away(off / dm), 0), 0, 15)
        s = np.repeat(dd * sc, 16)
        mu = np.repeat(dm * mm, 16)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away((w + mu) / s), 0.0)
        return {"q": np.clip(r, 0, 3).astype(np.uint8), "sc": sc.astype(np.uint8), "m": mm.astype(np.uint8),
                "d": d, "dmin": dmin}
    if fmt in (Q4_K, Q5_K):
        top = 15 if fmt == Q4_K else 31
        mn = np.minimum(blk.min(axis=1), 0.0)
        scale = (blk.max(axis=1) - mn) / top
        off = -mn
        sup_s = scale.reshape(-1, 8).max(axis=1)
        sup_o = off.reshape(-1, 8).max(axis=1)
        d = (sup_s / 63).astype(np.float16)
        dmin = (sup_o / 63).astype(np.float16)
        dd = np.repeat(d.astype(np.float64), 8)
        dm = np.repeat(dmin.astype(np.float64), 8)
        with np.errstate(divide="ignore", invalid="ignore"):
            sc = np.clip(np.where(dd > 0, _round_half_away(scale / dd), 0), 0, 63)
            mm = np.clip(np.where(dm > 0, _round_half_away(off / dm), 0), 0, 63)
        s = np.repeat(dd * sc, 32)
        mu = np.repeat(dm * mm, 32)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(s > 0, _round_half_away((w + mu) / s), 0.0)
        return {"q": np.clip(r, 0, top).astype(np.uint8), "sc": sc.astype(np.uint8), "m": mm.astype(np.uint8),
                "d": d, "dmin": dmin}
    raise ValueError(fmt)


def zero_rows(fmt: int, f: dict, rows, K: int) -> dict:
    """A copy of the fields in which every weight of the given rows (of a
    row-major matrix with K columns) is exactly zero while the rows' scales
    stay nonzero, chosen so that each row's codes and scales are those of the
    format's other blocks:
    q4_0  codes 8; q4_1  codes 4 and m = -4 d (exact in binary16);
    q4_k  codes 3, dmin = d and m_j = 3 sc_j (sc_j in [1, 21]);
    q8_0  codes 0; f16  +0; q1_0 has no zero level: its scales are set to 0;
    q5_0  codes 16; q5_1  codes 4 and m = -4 d; q5_k  as q4_k; q6_k  codes 32;
    q2_k  codes 3 with dmin = d and m_j = 3 sc_j (sc_j in [1, 5])."""
    f = {k: v.copy() for k, v in f.items()}
    rows = np.asarray(rows, np.int64)
    el = (rows[:, None] * K + np.arange(K)[None, :]).reshape(-1)
    grp = np.unique(el // 32)
    if fmt == F16:
        f["w"][el] = np.float16(0)
    elif fmt == Q8_0:
        f["q"][el] = 0
    elif fmt == Q4_0:
        f["q"][el] = 8
    elif fmt == Q4_1:
        f["q"][el] = 4
        f["m"][grp] = (-4.0 * f["d"][grp].astype(np.float64)).astype(np.float16)
    elif fmt == Q4_K:
        f["q"][el] = 3
        sup = np.unique(el // 256)
        f["dmin"][sup] = f["d"][sup]
        sc = (np.arange(grp.size) % 21 + 1).astype(np.uint8)
        f["sc"][grp] = sc
        f["m"][grp] = 3 * sc
    elif fmt == Q1_0:
        f["d"][np.unique(el // 128)] = np.float16(0)
    elif fmt == Q5_0:
        f["q"][el] = 16
    elif fmt == Q5_1:
        f["q"][el] = 4
        f["m"][grp] = (-4.0 * f["d"][grp].astype(np.float64)).astype(np.float16)
    elif fmt == Q5_K:
        f["q"][el] = 3
        sup = np.unique(el // 256)
        f["dmin"][sup] = f["d"][sup]
        sc = (np.arange(grp.size) % 21 + 1).astype(np.uint8)
        f["sc"][grp] = sc
        f["m"][grp] = 3 * sc
    elif fmt == Q6_K:
        f["q"][el] = 32
    elif fmt == MXFP4:
        f["q"][el] = np.where(np.arange(el.size) % 2 == 0, 0, 8)  # +0 and -0
    elif fmt == Q2_K:
        f["q"][el] = 3
        sup = np.unique(el // 256)
        f["dmin"][sup] = f["d"][sup]
        g16 = np.unique(el // 16)
        sc = (np.arange(g16.size) % 5 + 1).astype(np.uint8)
        f["sc"][g16] = sc
        f["m"][g16] = 3 * sc
    else:
        raise ValueError(fmt)
    return f


def zero_scales(fmt: int, f: dict, rng: np.random.Generator, frac: float = 0.25) -> dict:
    """A copy of the fields with a random fraction of the blocks' scales set
    to zero (q4_1, q5_1: d = 0, the min kept; the K-quants with a min: d = 0
    on some super-blocks, d and dmin = 0 on others). f16 is returned
    unchanged."""
    f = {k: v.copy() for k, v in f.items()}
    if fmt == F16:
        return f
    if fmt == MXFP4:
        # the smallest exponent: a block scale of 2^-127 (binary32 subnormal products)
        f["E"][rng.random(f["E"].size) < frac] = 0
        return f
    d = f["d"]
    pick = rng.random(d.size) < frac
    d[pick] = np.float16(0)
    if fmt in (Q4_K, Q5_K, Q2_K):
        both = pick & (rng.random(d.size) < 0.5)
        f["dmin"][both] = np.float16(0)
    return f
