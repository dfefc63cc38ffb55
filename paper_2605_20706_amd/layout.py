"""Packers for the lw split-plane weight layout (byte placement only).

These functions place already-quantized fields (codes, scales, mins) into the
byte layout that ``include/lw.h`` specifies; they compute no dequantized value
and no product. Users call them to lay out weights they quantized themselves;
the tests and the benchmark call them (through ``synth``) to build seeded
synthetic inputs that both the HIP library and the CPU oracle then read.

Layout summary (little-endian; each plane after the first starts at the end of
the previous one rounded up to 256 bytes):

* f16   plane 0: n x binary16
* q8_0  plane 0: n x int8 codes;   plane 1: n/32 x binary16 d
* q4_0  plane 0: n/2 bytes, group g owns bytes [16g, 16g+16), byte i holds
        element 32g+i (bits 0-3) and 32g+i+16 (bits 4-7);  plane 1: n/32 x binary16 d
* q4_k  plane 0: as q4_0;  plane 1: n/256 x 12-byte record, a 96-bit
        little-endian integer with sc_j at bits [6j, 6j+6) and m_j at bits
        [48+6j, 48+6j+6);  plane 2: n/256 x {binary16 d, binary16 dmin}
* q4_1  plane 0: as q4_0;  plane 1: n/32 x {binary16 d, binary16 m}
* q1_0  plane 0: n/8 bytes, element e at bit (e mod 8) of byte e/8;
        plane 1: n/128 x binary16 d
* q5_0  plane 0: the low four bits of each 5-bit code, as q4_0's plane 0;
        plane 1: n/8 bytes of fifth bits, element e at bit (e mod 8) of byte e/8;
        plane 2: n/32 x binary16 d
* q5_1  planes 0, 1 as q5_0;  plane 2: n/32 x {binary16 d, binary16 m}
* q5_k  planes 0, 1 as q5_0;  plane 2: the q4_k records;  plane 3: n/256 x {d, dmin}
* q6_k  plane 0: the low four bits of each 6-bit code, as q4_0's plane 0;
        plane 1: n/4 bytes of high two bits, element e at bits 2(e mod 4) of byte e/4;
        plane 2: n/16 x int8 scale (sub-block of 16);  plane 3: n/256 x binary16 d
* mxfp4 plane 0: 4-bit e2m1 codes (sign in bit 3), as q4_0's plane 0;
        plane 1: n/32 e8m0 exponent bytes E (value = e2m1 * 2^(E - 127))
* q2_k  plane 0: n/4 bytes of 2-bit codes, element e at bits 2(e mod 4) of byte e/4;
        plane 1: n/16 bytes, sub-block scale in bits 0-3 and min in bits 4-7;
        plane 2: n/256 x {binary16 d, binary16 dmin}
"""
from __future__ import annotations

import numpy as np

F16, Q8_0, Q4_0, Q4_K, Q4_1, Q1_0 = 0, 1, 2, 3, 4, 5
Q5_0, Q5_1, Q5_K, Q6_K, Q2_K, MXFP4 = 6, 7, 8, 9, 10, 11
FORMATS = {"f16": F16, "q8_0": Q8_0, "q4_0": Q4_0, "q4_k": Q4_K, "q4_1": Q4_1, "q1_0": Q1_0,
           "q5_0": Q5_0, "q5_1": Q5_1, "q5_k": Q5_K, "q6_k": Q6_K, "q2_k": Q2_K, "mxfp4": MXFP4}
FORMAT_NAMES = {v: k for k, v in FORMATS.items()}
# Packed bytes per weight (codes and scales, ignoring plane padding).
BYTES_PER_WEIGHT = {F16: 2.0, Q8_0: 34.0 / 32.0, Q4_0: 18.0 / 32.0, Q4_K: 144.0 / 256.0, Q4_1: 20.0 / 32.0,
                    Q1_0: 18.0 / 128.0, Q5_0: 22.0 / 32.0, Q5_1: 24.0 / 32.0, Q5_K: 176.0 / 256.0,
                    Q6_K: 210.0 / 256.0, Q2_K: 84.0 / 256.0, MXFP4: 17.0 / 32.0}

ALIGN = 256


def _up(v: int) -> int:
    return (v + ALIGN - 1) // ALIGN * ALIGN


def plane_offsets(fmt: int, n: int):
    """(offsets of planes 0..2, total bytes) for n elements (planes 0..3 for
    the formats with four planes: plane_offsets4)."""
    offs, total = plane_offsets4(fmt, n)
    if offs[3]:
        raise ValueError("format %d has four planes: use plane_offsets4" % fmt)
    return offs[:3], total


def plane_offsets4(fmt: int, n: int):
    """(offsets of planes 0..3, total bytes) for n elements."""
    if n < 0:
        raise ValueError("n < 0")
    if fmt in (Q5_0, Q5_1):
        if n % 32:
            raise ValueError("n must be a multiple of 32")
        o1 = _up(n // 2)
        o2 = _up(o1 + n // 8)
        return (0, o1, o2, 0), o2 + (2 if fmt == Q5_0 else 4) * (n // 32)
    if fmt in (Q5_K, Q6_K, Q2_K):
        if n % 256:
            raise ValueError("n must be a multiple of 256")
        if fmt == Q5_K:
            o1 = _up(n // 2)
            o2 = _up(o1 + n // 8)
            o3 = _up(o2 + 12 * (n // 256))
            return (0, o1, o2, o3), o3 + 4 * (n // 256)
        if fmt == Q6_K:
            o1 = _up(n // 2)
            o2 = _up(o1 + n // 4)
            o3 = _up(o2 + n // 16)
            return (0, o1, o2, o3), o3 + 2 * (n // 256)
        o1 = _up(n // 4)
        o2 = _up(o1 + n // 16)
        return (0, o1, o2, 0), o2 + 4 * (n // 256)
    offs, total = _plane_offsets3(fmt, n)
    return tuple(offs) + (0,), total


def _plane_offsets3(fmt: int, n: int):
    if fmt == F16:
        return (0, 0, 0), 2 * n
    if fmt in (Q8_0, Q4_0):
        if n % 32:
            raise ValueError("n must be a multiple of 32")
        o1 = _up(n if fmt == Q8_0 else n // 2)
        return (0, o1, 0), o1 + 2 * (n // 32)
    if fmt == Q4_1:
        if n % 32:
            raise ValueError("n must be a multiple of 32")
        o1 = _up(n // 2)
        return (0, o1, 0), o1 + 4 * (n // 32)
    if fmt == Q1_0:
        if n % 128:
            raise ValueError("n must be a multiple of 128")
        o1 = _up(n // 8)
        return (0, o1, 0), o1 + 2 * (n // 128)
    if fmt == MXFP4:
        if n % 32:
            raise ValueError("n must be a multiple of 32")
        o1 = _up(n // 2)
        return (0, o1, 0), o1 + n // 32
    if fmt == Q4_K:
        if n % 256:
            raise ValueError("n must be a multiple of 256")
        o1 = _up(n // 2)
        o2 = _up(o1 + 12 * (n // 256))
        return (0, o1, o2), o2 + 4 * (n // 256)
    raise ValueError("unknown format %r" % (fmt,))


def _half_bits(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.float16:
        return a.view(np.uint16).reshape(-1)
    if a.dtype == np.uint16:
        return a.reshape(-1)
    raise TypeError("binary16 fields must be float16 or uint16 bit patterns")


def pack_nibbles(q) -> np.ndarray:
    """4-bit codes (n,) in [0, 15] -> n/2 bytes in the group-of-32 nibble order."""
    q = np.asarray(q, dtype=np.uint8).reshape(-1, 2, 16)
    if q.size and int(q.max()) > 15:
        raise ValueError("4-bit codes must lie in [0, 15]")
    return (q[:, 0, :] | (q[:, 1, :] << 4)).reshape(-1)


def pack_q4k_records(sc, m) -> np.ndarray:
    """6-bit sub-block scales and mins, shape (n/32,) each, -> (n/256, 12) bytes."""
    sc = np.asarray(sc, dtype=np.uint64).reshape(-1, 8)
    m = np.asarray(m, dtype=np.uint64).reshape(-1, 8)
    if sc.size and (int(sc.max()) > 63 or int(m.max()) > 63):
        raise ValueError("6-bit fields must lie in [0, 63]")
    shifts = (np.arange(8, dtype=np.uint64) * np.uint64(6))
    lo = np.bitwise_or.reduce(sc << shifts, axis=1)  # bits 0..47 of R
    hi = np.bitwise_or.reduce(m << shifts, axis=1)   # bits 48..95 of R
    rec = np.empty((sc.shape[0], 12), dtype=np.uint8)
    rec[:, 0:6] = lo.astype("<u8").view(np.uint8).reshape(-1, 8)[:, 0:6]
    rec[:, 6:12] = hi.astype("<u8").view(np.uint8).reshape(-1, 8)[:, 0:6]
    return rec


def assemble(fmt: int, n: int, plane0: np.ndarray, plane1=None, plane2=None, plane3=None) -> np.ndarray:
    """Place already-encoded plane bytes at their offsets (zero padding)."""
    offs, total = plane_offsets4(fmt, n)
    out = np.zeros(total, dtype=np.uint8)
    for i, p in enumerate((plane0, plane1, plane2, plane3)):
        if p is None:
            continue
        p = np.ascontiguousarray(p).view(np.uint8).reshape(-1)
        out[offs[i]:offs[i] + p.size] = p
    return out


def pack_f16(w) -> np.ndarray:
    h = _half_bits(w).astype("<u2")
    return assemble(F16, h.size, h)


def pack_q8_0(q, d) -> np.ndarray:
    q = np.asarray(q)
    if q.dtype != np.int8:
        if q.size and (int(q.min()) < -128 or int(q.max()) > 127):
            raise ValueError("int8 codes out of range")
        q = q.astype(np.int8)
    q = q.reshape(-1)
    d = _half_bits(d).astype("<u2")
    if d.size * 32 != q.size:
        raise ValueError("need one scale per 32 codes")
    return assemble(Q8_0, q.size, q, d)


def pack_q4_0(q, d) -> np.ndarray:
    q = np.asarray(q).reshape(-1)
    d = _half_bits(d).astype("<u2")
    if d.size * 32 != q.size:
        raise ValueError("need one scale per 32 codes")
    return assemble(Q4_0, q.size, pack_nibbles(q), d)


def pack_q4_k(q, sc, m, d, dmin) -> np.ndarray:
    q = np.asarray(q).reshape(-1)
    n = q.size
    d = _half_bits(d)
    dmin = _half_bits(dmin)
    if d.size * 256 != n or dmin.size * 256 != n or np.size(sc) * 32 != n or np.size(m) * 32 != n:
        raise ValueError("q4_k field sizes do not match n")
    dd = np.empty((n // 256, 2), dtype="<u2")
    dd[:, 0] = d
    dd[:, 1] = dmin
    return assemble(Q4_K, n, pack_nibbles(q), pack_q4k_records(sc, m), dd)


def pack_q4_1(q, d, m) -> np.ndarray:
    q = np.asarray(q).reshape(-1)
    d = _half_bits(d)
    m = _half_bits(m)
    if d.size * 32 != q.size or m.size * 32 != q.size:
        raise ValueError("need one scale and one min per 32 codes")
    dm = np.empty((q.size // 32, 2), dtype="<u2")
    dm[:, 0] = d
    dm[:, 1] = m
    return assemble(Q4_1, q.size, pack_nibbles(q), dm)


def pack_bits(b) -> np.ndarray:
    """1-bit codes (n,) in {0, 1} -> n/8 bytes, element e at bit (e mod 8) of byte e/8."""
    b = np.asarray(b, dtype=np.uint8).reshape(-1)
    if b.size and int(b.max()) > 1:
        raise ValueError("1-bit codes must lie in {0, 1}")
    return np.packbits(b, bitorder="little")


def pack_q1_0(b, d) -> np.ndarray:
    b = np.asarray(b).reshape(-1)
    d = _half_bits(d).astype("<u2")
    if d.size * 128 != b.size:
        raise ValueError("need one scale per 128 codes")
    return assemble(Q1_0, b.size, pack_bits(b), d)


def pack_2bit(v) -> np.ndarray:
    """2-bit fields (n,) in [0, 3] -> n/4 bytes, element e at bits 2(e mod 4) of byte e/4."""
    v = np.asarray(v, dtype=np.uint8).reshape(-1, 4)
    if v.size and int(v.max()) > 3:
        raise ValueError("2-bit fields must lie in [0, 3]")
    return (v[:, 0] | (v[:, 1] << 2) | (v[:, 2] << 4) | (v[:, 3] << 6)).astype(np.uint8)


def _split5(q):
    q = np.asarray(q, dtype=np.uint8).reshape(-1)
    if q.size and int(q.max()) > 31:
        raise ValueError("5-bit codes must lie in [0, 31]")
    return pack_nibbles(q & 15), pack_bits(q >> 4)


def pack_q5_0(q, d) -> np.ndarray:
    q = np.asarray(q).reshape(-1)
    d = _half_bits(d).astype("<u2")
    if d.size * 32 != q.size:
        raise ValueError("need one scale per 32 codes")
    lo, hi = _split5(q)
    return assemble(Q5_0, q.size, lo, hi, d)


def pack_q5_1(q, d, m) -> np.ndarray:
    q = np.asarray(q).reshape(-1)
    d, m = _half_bits(d), _half_bits(m)
    if d.size * 32 != q.size or m.size * 32 != q.size:
        raise ValueError("need one scale and one min per 32 codes")
    dm = np.empty((q.size // 32, 2), dtype="<u2")
    dm[:, 0] = d
    dm[:, 1] = m
    lo, hi = _split5(q)
    return assemble(Q5_1, q.size, lo, hi, dm)


def pack_q5_k(q, sc, m, d, dmin) -> np.ndarray:
    q = np.asarray(q).reshape(-1)
    n = q.size
    d, dmin = _half_bits(d), _half_bits(dmin)
    if d.size * 256 != n or dmin.size * 256 != n or np.size(sc) * 32 != n or np.size(m) * 32 != n:
        raise ValueError("q5_k field sizes do not match n")
    dd = np.empty((n // 256, 2), dtype="<u2")
    dd[:, 0] = d
    dd[:, 1] = dmin
    lo, hi = _split5(q)
    return assemble(Q5_K, n, lo, hi, pack_q4k_records(sc, m), dd)


def pack_q6_k(q, sc, d) -> np.ndarray:
    """6-bit codes q (n,) in [0, 63], int8 scales sc (n/16,), binary16 d (n/256,)."""
    q = np.asarray(q, dtype=np.uint8).reshape(-1)
    n = q.size
    if q.size and int(q.max()) > 63:
        raise ValueError("6-bit codes must lie in [0, 63]")
    sc = np.asarray(sc)
    if sc.dtype != np.int8:
        if sc.size and (int(sc.min()) < -128 or int(sc.max()) > 127):
            raise ValueError("int8 scales out of range")
        sc = sc.astype(np.int8)
    d = _half_bits(d).astype("<u2")
    if d.size * 256 != n or sc.size * 16 != n:
        raise ValueError("q6_k field sizes do not match n")
    return assemble(Q6_K, n, pack_nibbles(q & 15), pack_2bit(q >> 4), sc.reshape(-1), d)


def pack_q2_k(q, sc, m, d, dmin) -> np.ndarray:
    """2-bit codes q (n,), 4-bit scales sc and mins m (n/16,), binary16 d and dmin (n/256,)."""
    q = np.asarray(q).reshape(-1)
    n = q.size
    sc = np.asarray(sc, dtype=np.uint8).reshape(-1)
    m = np.asarray(m, dtype=np.uint8).reshape(-1)
    if sc.size and (int(sc.max()) > 15 or int(m.max()) > 15):
        raise ValueError("4-bit scales and mins must lie in [0, 15]")
    d, dmin = _half_bits(d), _half_bits(dmin)
    if d.size * 256 != n or dmin.size * 256 != n or sc.size * 16 != n or m.size * 16 != n:
        raise ValueError("q2_k field sizes do not match n")
    dd = np.empty((n // 256, 2), dtype="<u2")
    dd[:, 0] = d
    dd[:, 1] = dmin
    return assemble(Q2_K, n, pack_2bit(q), (sc | (m << 4)).astype(np.uint8), dd)


def pack_mxfp4(codes, E) -> np.ndarray:
    """4-bit e2m1 codes (n,) in [0, 15] (bit 3 the sign) and e8m0 exponents
    (n/32,) in [0, 255] -> the mxfp4 layout."""
    codes = np.asarray(codes).reshape(-1)
    E = np.asarray(E, dtype=np.uint8).reshape(-1)
    if E.size * 32 != codes.size:
        raise ValueError("need one exponent per 32 codes")
    return assemble(MXFP4, codes.size, pack_nibbles(codes), E)
