"""CPU oracle for the fused dequantize x matrix-vector product.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path (the HIP library and
its Python binding) never does, and this package imports nothing from it.

The arithmetic lives in ``lw_oracle.c`` (plain scalar C, double precision, one
rounding per dequantized element, fixed summation order); this module only
builds it with gcc and marshals numpy arrays through ctypes.

* ``dequant(fmt, W_bytes, n)`` -> float32[n], the exact closed form of each
  element rounded once (Eq. (1) of Sec. 2.2 with the legacy and K-quant block
  structures of Sec. 2.2).
* ``matvec(fmt, W_bytes, x, M, K)`` -> (y, A) in float64: y = dequant(W) . x
  (Sec. 2.1: decode is a matrix-vector product) and A = sum_k |w * x|.
* ``matvec_f(fmt, W_bytes, x, M, K, beta)`` -> (y, A, F): also the term mass
  F of Eq. (1)'s two terms with the unsigned code shifted by beta,
  F = sum_k (|s|*(q + beta) + |mu - beta*s|) * |x| (F = A for f16 and q8_0),
  the quantity that scales the rounding error of a kernel that sums the two
  terms separately.
* ``matvec_sampled(...)`` the same for a list of (token, row) outputs.
* ``attn_decode(fmt, q, K, V, n_heads, n_kv_heads, head_dim, kv_len, scale)``
  -> (out, A, T): one query token's attention over a KV cache stored in a
  weight format (Sec. 3.2 attention over quantized K/V, Sec. 3.3 the
  dequantization reused for the KV cache), with A = sum_j p_j |v_j| per
  output and T = the largest scale * sum |q k| per head.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lw_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0 = 0, 1, 2, 3, 4, 5

_lib = None
# A test may point this module at another build of the oracle (a copy with a
# planted mistake) through the environment; the default is liboracle.so here.
_LIB_OVERRIDE = os.environ.get("LW_ORACLE_LIB")


def build(force: bool = True) -> str:
    """Compile lw_oracle.c into liboracle.so next to it (plain -O2, no FMA
    contraction, no fast-math, no vector intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
                               "-fPIC", "-shared", "-pthread", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            lib = ctypes.CDLL(_LIB)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        f32p = ctypes.POINTER(ctypes.c_float)
        f64p = ctypes.POINTER(ctypes.c_double)
        i64p = ctypes.POINTER(ctypes.c_int64)
        i64 = ctypes.c_int64
        lib.oracle_weight_bytes.argtypes = [ctypes.c_int, i64]
        lib.oracle_weight_bytes.restype = i64
        lib.oracle_dequant.argtypes = [ctypes.c_int, u8p, i64, f32p]
        lib.oracle_dequant.restype = ctypes.c_int
        lib.oracle_matvec.argtypes = [ctypes.c_int, u8p, f32p, i64, i64, i64, f64p, f64p, ctypes.c_int]
        lib.oracle_matvec.restype = ctypes.c_int
        lib.oracle_matvec_f.argtypes = [ctypes.c_int, u8p, f32p, i64, i64, i64, f64p, f64p, f64p, ctypes.c_int,
                                        ctypes.c_int]
        lib.oracle_matvec_f.restype = ctypes.c_int
        lib.oracle_matvec_sampled.argtypes = [ctypes.c_int, u8p, f32p, i64, i64, i64, i64,
                                              i64p, i64p, f64p, f64p]
        lib.oracle_matvec_sampled.restype = ctypes.c_int
        lib.oracle_attn_decode.argtypes = [ctypes.c_int, f32p, u8p, u8p, i64, i64, i64, i64, ctypes.c_double,
                                           f64p, f64p, f64p]
        lib.oracle_attn_decode.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _bytes(W) -> np.ndarray:
    W = np.ascontiguousarray(W)
    if W.dtype != np.uint8:
        W = W.view(np.uint8)
    return W.reshape(-1)


def weight_bytes(fmt: int, n: int) -> int:
    return int(_load().oracle_weight_bytes(fmt, n))


def dequant(fmt: int, W, n: int) -> np.ndarray:
    W = _bytes(W)
    need = weight_bytes(fmt, n)
    if need < 0 or W.size < need:
        raise ValueError("oracle.dequant: bad format/size (need %d bytes, got %d)" % (need, W.size))
    out = np.empty(n, dtype=np.float32)
    if _load().oracle_dequant(fmt, _ptr(W, ctypes.c_uint8), n, _ptr(out, ctypes.c_float)) != 0:
        raise ValueError("oracle.dequant failed")
    return out


def matvec(fmt: int, W, x: np.ndarray, M: int, K: int, n_threads: int = 0):
    """Returns (y, A, threads): float64 arrays of shape [n_tok, M] and the
    number of threads used."""
    W = _bytes(W)
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x.reshape(1, -1)
    n_tok = x.shape[0]
    if x.shape[1] != K:
        raise ValueError("oracle.matvec: x has %d columns, K = %d" % (x.shape[1], K))
    need = weight_bytes(fmt, M * K)
    if need < 0 or W.size < need:
        raise ValueError("oracle.matvec: bad format/size")
    y = np.empty((n_tok, M), dtype=np.float64)
    A = np.empty((n_tok, M), dtype=np.float64)
    T = _load().oracle_matvec(fmt, _ptr(W, ctypes.c_uint8), _ptr(x, ctypes.c_float), M, K, n_tok,
                              _ptr(y, ctypes.c_double), _ptr(A, ctypes.c_double), n_threads)
    if T < 0:
        raise ValueError("oracle.matvec failed")
    return y, A, T


def matvec_f(fmt: int, W, x: np.ndarray, M: int, K: int, beta: int = 0, n_threads: int = 0):
    """Returns (y, A, F, threads): y and A as matvec's, F the term mass with
    code shift beta (0 <= beta <= 1024), all float64 [n_tok, M]."""
    W = _bytes(W)
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x.reshape(1, -1)
    n_tok = x.shape[0]
    if x.shape[1] != K:
        raise ValueError("oracle.matvec_f: x has %d columns, K = %d" % (x.shape[1], K))
    need = weight_bytes(fmt, M * K)
    if need < 0 or W.size < need:
        raise ValueError("oracle.matvec_f: bad format/size")
    y = np.empty((n_tok, M), dtype=np.float64)
    A = np.empty((n_tok, M), dtype=np.float64)
    F = np.empty((n_tok, M), dtype=np.float64)
    T = _load().oracle_matvec_f(fmt, _ptr(W, ctypes.c_uint8), _ptr(x, ctypes.c_float), M, K, n_tok,
                                _ptr(y, ctypes.c_double), _ptr(A, ctypes.c_double), _ptr(F, ctypes.c_double),
                                int(beta), n_threads)
    if T < 0:
        raise ValueError("oracle.matvec_f failed")
    return y, A, F, T


def matvec_sampled(fmt: int, W, x: np.ndarray, M: int, K: int, rows, toks):
    """y[s], A[s] for the outputs (toks[s], rows[s])."""
    W = _bytes(W)
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x.reshape(1, -1)
    n_tok = x.shape[0]
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    toks = np.ascontiguousarray(toks, dtype=np.int64)
    if rows.shape != toks.shape:
        raise ValueError("rows and toks differ in shape")
    need = weight_bytes(fmt, M * K)
    if need < 0 or W.size < need:
        raise ValueError("oracle.matvec_sampled: bad format/size")
    y = np.empty(rows.size, dtype=np.float64)
    A = np.empty(rows.size, dtype=np.float64)
    rc = _load().oracle_matvec_sampled(fmt, _ptr(W, ctypes.c_uint8), _ptr(x, ctypes.c_float), M, K,
                                       n_tok, rows.size, _ptr(rows, ctypes.c_int64),
                                       _ptr(toks, ctypes.c_int64), _ptr(y, ctypes.c_double),
                                       _ptr(A, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle.matvec_sampled failed")
    return y, A


def attn_decode(fmt: int, q, Kc, Vc, n_heads: int, n_kv_heads: int, head_dim: int, kv_len: int, scale: float):
    """Returns (out [n_heads, head_dim], A [n_heads, head_dim], T [n_heads]) in float64."""
    q = np.ascontiguousarray(q, dtype=np.float32).reshape(-1)
    if q.size != n_heads * head_dim:
        raise ValueError("oracle.attn_decode: q must hold n_heads * head_dim floats")
    Kc, Vc = _bytes(Kc), _bytes(Vc)
    need = weight_bytes(fmt, n_kv_heads * kv_len * head_dim)
    if need < 0 or Kc.size < need or Vc.size < need:
        raise ValueError("oracle.attn_decode: bad format/size")
    out = np.empty((n_heads, head_dim), np.float64)
    A = np.empty((n_heads, head_dim), np.float64)
    T = np.empty(n_heads, np.float64)
    rc = _load().oracle_attn_decode(fmt, _ptr(q, ctypes.c_float), _ptr(Kc, ctypes.c_uint8), _ptr(Vc, ctypes.c_uint8),
                                    n_heads, n_kv_heads, head_dim, kv_len, float(scale), _ptr(out, ctypes.c_double),
                                    _ptr(A, ctypes.c_double), _ptr(T, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle.attn_decode failed")
    return out, A, T
