/*
 * CPU oracle for the fused dequantize x matrix-vector product.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path links, loads or calls
 * this file; only the tests, the smoke check and the benchmark's CPU-baseline
 * leg do. It shares no code, header or table with the HIP library: it has its
 * own plane arithmetic, its own binary16 decoder and its own bit extraction.
 *
 * What it computes is the plain definition, written out slowly:
 *   - dequantization, one element at a time: read the fields of the element
 *     from the packed bytes, evaluate the closed form exactly in double
 *     precision (every product involved is exact there), and round once to
 *     float with the C cast (round to nearest, ties to even);
 *   - the matrix-vector product y[t][r] = sum_k w[r][k] * x[t][k] with
 *     w = the float dequantized weight, every product taken in double (exact:
 *     24 + 24 bits) and summed in double in the order k = 0, 1, ..., K-1;
 *     alongside it the condition sum A[t][r] = sum_k |w[r][k] * x[t][k]|;
 *   - optionally the term mass F[t][r] of the same product written with
 *     Eq. (1)'s two terms, value = s*q + mu for the stored unsigned code q,
 *     and the code shifted by a constant beta:
 *       value = s*(q + beta) + (mu - beta*s),
 *       F[t][r] = sum_k (|s_k|*(q_k + beta) + |mu_k - beta*s_k|) * |x[t][k]|.
 *     A kernel that sums the two terms separately (a factored form) rounds
 *     sums of these magnitudes, so F scales its rounding error the way A
 *     scales a plain sum's. Formats without an unsigned code and an offset
 *     (f16, q8_0) have F = A.
 *
 * Passages followed:
 *   - Eq. (1), Sec. 2.2: x_hat = s * q + mu (scale s, optional offset mu).
 *   - Sec. 2.2, legacy formats: blocks of 32 weights; q8_0 and q4_0 are
 *     symmetric (no offset): value = d * q for q8_0, d * (q - 8) for the
 *     unsigned 4-bit codes of q4_0.
 *   - Sec. 2.2, legacy formats with an offset (q4_1 among them): Eq. (1) with
 *     both terms per block of 32, scale d and offset (min) m stored as
 *     binary16: value = d * q + m for the unsigned 4-bit codes.
 *   - Sec. 2.2, K-quants: super-blocks of 256 = 8 sub-blocks of 32, each with
 *     its own scale, the scales quantized against a super-block scale; the
 *     K-quant style used here also carries a per-sub-block min quantized
 *     against a super-block dmin (Eq. (1)'s offset mu = -dmin * m):
 *     value = d * sc_j * q - dmin * m_j.
 *   - Sec. 2.2, q1_0: symmetric quantization with one scale per block of 128
 *     weights and one bit per weight; with Eq. (1)'s offset zero the bit b
 *     selects one of the two symmetric levels, q = 2b - 1, so value = +-d
 *     with the binary16 scale d of the block.
 *   - Sec. 2.2, 5-bit legacy formats (q5_0 symmetric, q5_1 with a min):
 *     blocks of 32, value = d * (q - 16) and d * q + m for 5-bit codes.
 *   - Sec. 2.2, further K-quants over super-blocks of 256 (Sec. 7 studies
 *     q2_k; Appendix B lists q2_k .. q6_k): q5_K-style as q4_K with 5-bit
 *     codes; q6_K-style with 16 sub-blocks of 16, a signed 8-bit scale each
 *     and one binary16 d, value = d * sc_j * (q - 32) for 6-bit codes;
 *     q2_K-style with 16 sub-blocks of 16, a 4-bit scale and a 4-bit min
 *     each against binary16 d and dmin, value = d * sc_j * q - dmin * m_j
 *     for 2-bit codes.
 *   - Sec. 2.2 and Appendix B, mxfp4 (the microscaling 4-bit float format
 *     the paper emulates for gpt-oss): blocks of 32 elements, each a 4-bit
 *     float e2m1 (sign, 2-bit exponent with bias 1, 1-bit mantissa: the
 *     magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6), sharing an 8-bit power-of-two
 *     scale E (e8m0): value = e2m1(code) * 2^(E - 127); E = 255 encodes NaN.
 *   - Sec. 2.1: decode is a matrix-vector product.
 *
 * Byte layout (the library's split-plane layout): plane 0 at offset 0; each
 * next plane at the end of the previous rounded up to 256 bytes; fields are
 * little-endian. Q4 nibbles: byte i of group g holds element 32g+i in its low
 * four bits and element 32g+i+16 in its high four bits. Q4_K plane 1 holds one
 * 12-byte record per super-block, read as a 96-bit little-endian integer R:
 * sc_j = bits [6j, 6j+6), m_j = bits [48+6j, 48+6j+6). Q4_K plane 2 holds
 * {binary16 d, binary16 dmin} per super-block. Q4_1 plane 0 is as Q4_0's;
 * plane 1 holds {binary16 d, binary16 m} per group of 32. Q1_0 plane 0 holds
 * one bit per element, element e at bit (e mod 8) of byte e/8; plane 1 holds
 * one binary16 d per block of 128.
 * The 5-bit formats keep the Q4 nibble plane for the low four bits of each
 * code and add a plane of fifth bits, element e at bit (e mod 8) of byte
 * e/8; then q5_0: binary16 d per 32; q5_1: {d, m} per 32; q5_K: the q4_K
 * record plane, then {d, dmin}. q6_K: the nibble plane for the low four
 * bits, a plane of the high two bits (element e at bits 2(e mod 4) of byte
 * e/4), one int8 scale per 16 elements, one binary16 d per 256. q2_K: the
 * 2-bit codes (element e at bits 2(e mod 4) of byte e/4), one byte per 16
 * elements with the scale in bits 0-3 and the min in bits 4-7, then
 * {d, dmin} per 256. mxfp4: the Q4 nibble plane of 4-bit codes, then one
 * e8m0 byte per 32 elements.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared -pthread (no fast-math, no
 * vector intrinsics). Results do not depend on the thread count: each output
 * has one fixed summation order.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

enum {
    OR_F16 = 0, OR_Q8_0 = 1, OR_Q4_0 = 2, OR_Q4_K = 3, OR_Q4_1 = 4, OR_Q1_0 = 5,
    OR_Q5_0 = 6, OR_Q5_1 = 7, OR_Q5_K = 8, OR_Q6_K = 9, OR_Q2_K = 10, OR_MXFP4 = 11
};

/* Elements per block: a row of K elements starts a block when K is a multiple. */
static int64_t block_elems(int fmt) {
    switch (fmt) {
    case OR_F16: return 1;
    case OR_Q4_K:
    case OR_Q5_K:
    case OR_Q6_K:
    case OR_Q2_K: return 256;
    case OR_Q1_0: return 128;
    default: return 32;
    }
}

/* ---- plane arithmetic ---------------------------------------------------- */

static int64_t round_up_256(int64_t v) { return (v + 255) / 256 * 256; }

/* Byte offset of each plane and the total size, for n elements of fmt.
 * Returns 0 on success, -1 for an unknown format or an n the format cannot
 * hold (negative, or not a multiple of the format's block). */
static int planes(int fmt, int64_t n, int64_t off[4], int64_t* total) {
    if (n < 0) return -1;
    off[0] = off[1] = off[2] = off[3] = 0;
    switch (fmt) {
    case OR_F16:
        *total = 2 * n;
        return 0;
    case OR_Q8_0:
        if (n % 32) return -1;
        off[1] = round_up_256(n);               /* n int8 codes */
        *total = off[1] + 2 * (n / 32);         /* n/32 binary16 scales */
        return 0;
    case OR_Q4_0:
        if (n % 32) return -1;
        off[1] = round_up_256(n / 2);           /* two codes per byte */
        *total = off[1] + 2 * (n / 32);
        return 0;
    case OR_Q4_1:
        if (n % 32) return -1;
        off[1] = round_up_256(n / 2);
        *total = off[1] + 4 * (n / 32);         /* n/32 {binary16 d, binary16 m} */
        return 0;
    case OR_Q1_0:
        if (n % 128) return -1;
        off[1] = round_up_256(n / 8);           /* one bit per element */
        *total = off[1] + 2 * (n / 128);        /* n/128 binary16 scales */
        return 0;
    case OR_Q4_K:
        if (n % 256) return -1;
        off[1] = round_up_256(n / 2);
        off[2] = round_up_256(off[1] + 12 * (n / 256));
        *total = off[2] + 4 * (n / 256);
        return 0;
    case OR_Q5_0:
    case OR_Q5_1:
        if (n % 32) return -1;
        off[1] = round_up_256(n / 2);            /* low four bits, two codes per byte */
        off[2] = round_up_256(off[1] + n / 8);   /* fifth bits, eight per byte */
        *total = off[2] + (fmt == OR_Q5_0 ? 2 : 4) * (n / 32);
        return 0;
    case OR_Q5_K:
        if (n % 256) return -1;
        off[1] = round_up_256(n / 2);
        off[2] = round_up_256(off[1] + n / 8);
        off[3] = round_up_256(off[2] + 12 * (n / 256));
        *total = off[3] + 4 * (n / 256);
        return 0;
    case OR_Q6_K:
        if (n % 256) return -1;
        off[1] = round_up_256(n / 2);            /* low four bits */
        off[2] = round_up_256(off[1] + n / 4);   /* high two bits, four codes per byte */
        off[3] = round_up_256(off[2] + n / 16);  /* int8 scale per 16 */
        *total = off[3] + 2 * (n / 256);         /* binary16 d per 256 */
        return 0;
    case OR_MXFP4:
        if (n % 32) return -1;
        off[1] = round_up_256(n / 2);            /* 4-bit codes, two per byte */
        *total = off[1] + n / 32;                /* one e8m0 exponent per 32 */
        return 0;
    case OR_Q2_K:
        if (n % 256) return -1;
        off[1] = round_up_256(n / 4);            /* 2-bit codes, four per byte */
        off[2] = round_up_256(off[1] + n / 16);  /* {scale, min} nibbles per 16 */
        *total = off[2] + 4 * (n / 256);         /* {d, dmin} per 256 */
        return 0;
    default:
        return -1;
    }
}

int64_t oracle_weight_bytes(int fmt, int64_t n) {
    int64_t off[4], total;
    if (planes(fmt, n, off, &total)) return -1;
    return total;
}

/* ---- field readers ------------------------------------------------------- */

static unsigned read_u16(const uint8_t* p) { return (unsigned)p[0] | ((unsigned)p[1] << 8); }

/* Exact real value of an IEEE 754 binary16 bit pattern, as a double.
 * sign | 5-bit exponent e | 10-bit fraction f:
 *   e = 0       subnormal or zero: f * 2^-24
 *   e = 31      infinity (f = 0) or NaN
 *   otherwise   (1024 + f) * 2^(e - 25)  (= (1 + f/1024) * 2^(e - 15)) */
static double half_value(unsigned h) {
    unsigned sign = (h >> 15) & 1u, e = (h >> 10) & 31u, f = h & 1023u;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024u + f), (int)e - 25);
    return sign ? -v : v;
}

/* Bit field [start, start+len) of a little-endian byte string, one bit at a time. */
static unsigned bit_field(const uint8_t* bytes, int start, int len) {
    unsigned v = 0;
    for (int b = 0; b < len; ++b) {
        int pos = start + b;
        unsigned bit = (bytes[pos / 8] >> (pos % 8)) & 1u;
        v |= bit << b;
    }
    return v;
}

/* 4-bit code of element e in a Q4 code plane. */
static unsigned q4_code(const uint8_t* codes, int64_t e) {
    int64_t g = e / 32;
    int i = (int)(e % 32);
    uint8_t byte = codes[16 * g + (i % 16)];
    return i < 16 ? (byte & 15u) : (byte >> 4);
}

/* 5-bit code of element e: the Q4 nibble (low four bits) plus the fifth bit
 * from its plane (element e at bit e mod 8 of byte e/8). */
static unsigned q5_code(const uint8_t* W, const int64_t off[4], int64_t e) {
    unsigned hi = bit_field(W + off[1] + e / 8, (int)(e % 8), 1);
    return q4_code(W, e) | (hi << 4);
}

/* 2-bit field of element e in a plane of four codes per byte (element e at
 * bits 2(e mod 4) of byte e/4). */
static unsigned two_bits(const uint8_t* plane, int64_t e) {
    return bit_field(plane + e / 4, 2 * (int)(e % 4), 2);
}

/* 6-bit code of element e of a q6_K-style tensor: the Q4 nibble plus the high
 * two bits from plane 1. */
static unsigned q6_code(const uint8_t* W, const int64_t off[4], int64_t e) {
    return q4_code(W, e) | (two_bits(W + off[1], e) << 4);
}

/* Magnitude of a 4-bit e2m1 float (bits 0-2 of the code; bit 3 is the sign):
 * exponent field e (bits 1-2, bias 1), mantissa bit m (bit 0); e = 0 is the
 * subnormal m * 2^-1, otherwise 2^(e - 1) * (1 + m/2). */
static double e2m1_magnitude(unsigned code) {
    unsigned e = (code >> 1) & 3u, m = code & 1u;
    if (e == 0) return 0.5 * (double)m;
    return ldexp(1.0 + 0.5 * (double)m, (int)e - 1);
}

/* ---- dequantization: exact closed form, one rounding ---------------------- */

/* The exact real value of element e (before the final rounding). */
static double exact_value(int fmt, const uint8_t* W, const int64_t off[4], int64_t e) {
    switch (fmt) {
    case OR_F16:
        return half_value(read_u16(W + 2 * e));
    case OR_Q8_0: {
        int q = (int)(int8_t)W[e];
        double d = half_value(read_u16(W + off[1] + 2 * (e / 32)));
        return (double)q * d; /* <= 8 + 11 significant bits: exact */
    }
    case OR_Q4_0: {
        int q = (int)q4_code(W, e);
        double d = half_value(read_u16(W + off[1] + 2 * (e / 32)));
        return (double)(q - 8) * d; /* exact */
    }
    case OR_Q4_1: {
        int q = (int)q4_code(W, e);
        double d = half_value(read_u16(W + off[1] + 4 * (e / 32)));
        double m = half_value(read_u16(W + off[1] + 4 * (e / 32) + 2));
        /* d*q has <= 15 significant bits; d*q and m are integer multiples of
         * 2^-24 below 2^20 in magnitude, so their double sum is exact */
        return (double)q * d + m;
    }
    case OR_Q1_0: {
        /* symmetric, two levels: code bit b stands for q = 2b - 1 */
        int b = (W[e / 8] >> (e % 8)) & 1;
        double d = half_value(read_u16(W + off[1] + 2 * (e / 128)));
        return (double)(2 * b - 1) * d; /* +-d: exact */
    }
    case OR_Q4_K: {
        int64_t S = e / 256;
        int j = (int)((e / 32) % 8);
        const uint8_t* rec = W + off[1] + 12 * S;
        unsigned sc = bit_field(rec, 6 * j, 6);
        unsigned m = bit_field(rec, 48 + 6 * j, 6);
        double d = half_value(read_u16(W + off[2] + 4 * S));
        double dmin = half_value(read_u16(W + off[2] + 4 * S + 2));
        unsigned q = q4_code(W, e);
        /* d*sc*q has <= 21 significant bits and dmin*m <= 17; for any finite
         * binary16 d and dmin the two lie within 2^26 .. 2^-24 of each other,
         * so the double difference below is exact as well. */
        double a = d * (double)sc * (double)q;
        double b = dmin * (double)m;
        return a - b;
    }
    case OR_Q5_0: {
        int q = (int)q5_code(W, off, e);
        double d = half_value(read_u16(W + off[2] + 2 * (e / 32)));
        return (double)(q - 16) * d; /* <= 5 + 11 significant bits: exact */
    }
    case OR_Q5_1: {
        int q = (int)q5_code(W, off, e);
        double d = half_value(read_u16(W + off[2] + 4 * (e / 32)));
        double m = half_value(read_u16(W + off[2] + 4 * (e / 32) + 2));
        return (double)q * d + m; /* both multiples of 2^-24 below 2^21: exact */
    }
    case OR_Q5_K: {
        int64_t S = e / 256;
        int j = (int)((e / 32) % 8);
        const uint8_t* rec = W + off[2] + 12 * S;
        unsigned sc = bit_field(rec, 6 * j, 6);
        unsigned m = bit_field(rec, 48 + 6 * j, 6);
        double d = half_value(read_u16(W + off[3] + 4 * S));
        double dmin = half_value(read_u16(W + off[3] + 4 * S + 2));
        unsigned q = q5_code(W, off, e);
        double a = d * (double)sc * (double)q; /* <= 22 significant bits */
        double b = dmin * (double)m;
        return a - b;
    }
    case OR_Q6_K: {
        int q = (int)q6_code(W, off, e);
        int sc = (int)(int8_t)W[off[2] + e / 16];
        double d = half_value(read_u16(W + off[3] + 2 * (e / 256)));
        /* |sc| <= 2^7 and |q - 32| <= 2^5: <= 23 significant bits, exact in
         * float as well */
        return d * (double)sc * (double)(q - 32);
    }
    case OR_MXFP4: {
        unsigned c = q4_code(W, e);
        unsigned E = W[off[1] + e / 32];
        if (E == 255) return NAN;
        double v = e2m1_magnitude(c) * ldexp(1.0, (int)E - 127); /* exact in double */
        return (c & 8u) ? -v : v;
    }
    case OR_Q2_K: {
        int64_t S = e / 256;
        unsigned q = two_bits(W, e);
        unsigned scm = W[off[1] + e / 16];
        unsigned sc = scm & 15u, m = scm >> 4;
        double d = half_value(read_u16(W + off[2] + 4 * S));
        double dmin = half_value(read_u16(W + off[2] + 4 * S + 2));
        double a = d * (double)sc * (double)q; /* <= 17 significant bits */
        double b = dmin * (double)m;
        return a - b;
    }
    default:
        return NAN;
    }
}

/* |s|*(q + beta) + |mu - beta*s| of element e, exact in double: Eq. (1)'s
 * scale s and offset mu of the element with its stored unsigned code q
 * (q4_0: s = d, mu = -8d; q4_1: s = d, mu = m; q4_K-style: s = d*sc_j,
 * mu = -dmin*m_j; q1_0: value = (2b - 1)*d, so s = 2d, q = b, mu = -d;
 * q5_0: s = d, mu = -16d; q5_1: s = d, mu = m; q5_K-style as q4_K;
 * q6_K-style: s = d*sc_j, mu = -32 s; q2_K-style: s = d*sc_j, mu = -dmin*m_j).
 * f16 and q8_0 have no offset term: the magnitude of the value itself. */
static double term_mass(int fmt, const uint8_t* W, const int64_t off[4], int64_t e, int beta) {
    double s, mu, q;
    switch (fmt) {
    case OR_Q4_0:
        s = half_value(read_u16(W + off[1] + 2 * (e / 32)));
        mu = -8.0 * s;
        q = (double)q4_code(W, e);
        break;
    case OR_Q4_1:
        s = half_value(read_u16(W + off[1] + 4 * (e / 32)));
        mu = half_value(read_u16(W + off[1] + 4 * (e / 32) + 2));
        q = (double)q4_code(W, e);
        break;
    case OR_Q1_0: {
        double d = half_value(read_u16(W + off[1] + 2 * (e / 128)));
        s = 2.0 * d;
        mu = -d;
        q = (double)((W[e / 8] >> (e % 8)) & 1);
        break;
    }
    case OR_Q4_K: {
        int64_t S = e / 256;
        int j = (int)((e / 32) % 8);
        const uint8_t* rec = W + off[1] + 12 * S;
        s = half_value(read_u16(W + off[2] + 4 * S)) * (double)bit_field(rec, 6 * j, 6);
        mu = -half_value(read_u16(W + off[2] + 4 * S + 2)) * (double)bit_field(rec, 48 + 6 * j, 6);
        q = (double)q4_code(W, e);
        break;
    }
    case OR_Q5_0:
        s = half_value(read_u16(W + off[2] + 2 * (e / 32)));
        mu = -16.0 * s;
        q = (double)q5_code(W, off, e);
        break;
    case OR_Q5_1:
        s = half_value(read_u16(W + off[2] + 4 * (e / 32)));
        mu = half_value(read_u16(W + off[2] + 4 * (e / 32) + 2));
        q = (double)q5_code(W, off, e);
        break;
    case OR_Q5_K: {
        int64_t S = e / 256;
        int j = (int)((e / 32) % 8);
        const uint8_t* rec = W + off[2] + 12 * S;
        s = half_value(read_u16(W + off[3] + 4 * S)) * (double)bit_field(rec, 6 * j, 6);
        mu = -half_value(read_u16(W + off[3] + 4 * S + 2)) * (double)bit_field(rec, 48 + 6 * j, 6);
        q = (double)q5_code(W, off, e);
        break;
    }
    case OR_Q6_K:
        s = half_value(read_u16(W + off[3] + 2 * (e / 256))) * (double)(int8_t)W[off[2] + e / 16];
        mu = -32.0 * s;
        q = (double)q6_code(W, off, e);
        break;
    case OR_Q2_K: {
        int64_t S = e / 256;
        unsigned scm = W[off[1] + e / 16];
        s = half_value(read_u16(W + off[2] + 4 * S)) * (double)(scm & 15u);
        mu = -half_value(read_u16(W + off[2] + 4 * S + 2)) * (double)(scm >> 4);
        q = (double)two_bits(W, e);
        break;
    }
    default:
        return fabs((double)(float)exact_value(fmt, W, off, e));
    }
    /* s has <= 19 significant bits and q + beta <= 2^11: the products and
     * the difference below are exact in double for the scales of every
     * finite binary16 */
    return fabs(s) * (q + (double)beta) + fabs(mu - (double)beta * s);
}

/* out[e] = float(value(e)) for e in [0, n). Returns 0, or -1 on a bad
 * format or n. Single-threaded. */
int oracle_dequant(int fmt, const uint8_t* W, int64_t n, float* out) {
    int64_t off[4], total;
    if (planes(fmt, n, off, &total)) return -1;
    for (int64_t e = 0; e < n; ++e) out[e] = (float)exact_value(fmt, W, off, e);
    return 0;
}

/* ---- matrix-vector product ------------------------------------------------ */

typedef struct {
    int fmt;
    const uint8_t* W;
    const int64_t* off;
    const float* x;
    int64_t M, K, n_tok;
    double* y;
    double* A;
    double* F;
    int beta;
    int64_t r_begin, r_end;
} mv_job;

static void* mv_rows(void* arg) {
    mv_job* jb = (mv_job*)arg;
    float* w = (float*)malloc(sizeof(float) * (size_t)jb->K);
    double* tm = jb->F ? (double*)malloc(sizeof(double) * (size_t)jb->K) : NULL;
    if (!w || (jb->F && !tm)) {
        free(w);
        free(tm);
        return (void*)1;
    }
    for (int64_t r = jb->r_begin; r < jb->r_end; ++r) {
        /* the row of dequantized weights, each rounded once to float */
        for (int64_t k = 0; k < jb->K; ++k)
            w[k] = (float)exact_value(jb->fmt, jb->W, jb->off, r * jb->K + k);
        if (tm)
            for (int64_t k = 0; k < jb->K; ++k) tm[k] = term_mass(jb->fmt, jb->W, jb->off, r * jb->K + k, jb->beta);
        for (int64_t t = 0; t < jb->n_tok; ++t) {
            const float* xt = jb->x + t * jb->K;
            double s = 0.0, a = 0.0;
            for (int64_t k = 0; k < jb->K; ++k) {
                double p = (double)w[k] * (double)xt[k]; /* exact in double */
                s += p;
                a += fabs(p);
            }
            jb->y[t * jb->M + r] = s;
            if (jb->A) jb->A[t * jb->M + r] = a;
            if (tm) {
                double f = 0.0;
                for (int64_t k = 0; k < jb->K; ++k) f += tm[k] * fabs((double)xt[k]);
                jb->F[t * jb->M + r] = f;
            }
        }
    }
    free(w);
    free(tm);
    return NULL;
}

static int n_threads_or_default(int n_threads) {
    if (n_threads > 0) return n_threads;
    long c = sysconf(_SC_NPROCESSORS_ONLN);
    return c > 0 ? (int)c : 1;
}

/* y[t*M + r], A[t*M + r] and F[t*M + r] (A, F may be NULL; F with code
 * shift beta, 0 <= beta <= 1024) for all t < n_tok, r < M. x is float
 * [n_tok][K]. n_threads <= 0 uses every online CPU. Returns the number of
 * threads used, or -1 on a bad argument / allocation failure. */
int oracle_matvec_f(int fmt, const uint8_t* W, const float* x, int64_t M, int64_t K,
                    int64_t n_tok, double* y, double* A, double* F, int beta, int n_threads) {
    int64_t off[4], total;
    if (M < 1 || K < 1 || n_tok < 1 || !W || !x || !y || beta < 0 || beta > 1024) return -1;
    if (planes(fmt, M * K, off, &total) || K % block_elems(fmt)) return -1;
    int T = n_threads_or_default(n_threads);
    if (T > M) T = (int)M;
    pthread_t* th = (pthread_t*)calloc((size_t)T, sizeof(pthread_t));
    mv_job* jobs = (mv_job*)calloc((size_t)T, sizeof(mv_job));
    if (!th || !jobs) {
        free(th);
        free(jobs);
        return -1;
    }
    int failed = 0;
    for (int i = 0; i < T; ++i) {
        mv_job jb = {fmt, W, off, x, M, K, n_tok, y, A, F, beta, M * i / T, M * (i + 1) / T};
        jobs[i] = jb;
        if (pthread_create(&th[i], NULL, mv_rows, &jobs[i])) {
            mv_rows(&jobs[i]); /* could not start a thread: do its rows here */
            th[i] = 0;
        }
    }
    for (int i = 0; i < T; ++i) {
        void* rv = NULL;
        if (th[i]) pthread_join(th[i], &rv);
        if (rv) failed = 1;
    }
    free(th);
    free(jobs);
    return failed ? -1 : T;
}

/* oracle_matvec_f without the term mass. */
int oracle_matvec(int fmt, const uint8_t* W, const float* x, int64_t M, int64_t K,
                  int64_t n_tok, double* y, double* A, int n_threads) {
    return oracle_matvec_f(fmt, W, x, M, K, n_tok, y, A, NULL, 0, n_threads);
}

/* The same product for a list of single outputs: for s < n_samples,
 * y[s] = y_full[toks[s]][rows[s]] and A[s] likewise (A may be NULL).
 * Single-threaded. Returns 0 or -1. */
int oracle_matvec_sampled(int fmt, const uint8_t* W, const float* x, int64_t M, int64_t K,
                          int64_t n_tok, int64_t n_samples, const int64_t* rows,
                          const int64_t* toks, double* y, double* A) {
    int64_t off[4], total;
    if (M < 1 || K < 1 || n_tok < 1 || !W || !x || !y || n_samples < 0) return -1;
    if (planes(fmt, M * K, off, &total) || K % block_elems(fmt)) return -1;
    for (int64_t s = 0; s < n_samples; ++s) {
        int64_t r = rows[s], t = toks[s];
        if (r < 0 || r >= M || t < 0 || t >= n_tok) return -1;
        const float* xt = x + t * K;
        double sum = 0.0, a = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double p = (double)(float)exact_value(fmt, W, off, r * K + k) * (double)xt[k];
            sum += p;
            a += fabs(p);
        }
        y[s] = sum;
        if (A) A[s] = a;
    }
    return 0;
}

/* ---- decode attention over a quantized KV cache ---------------------------
 *
 * Sec. 3.2 (attention kernels read quantized K and V and dequantize them on
 * load) and Sec. 3.3 (the dequantization routines serve the KV cache too).
 * One query token: for query head h and its key/value head g = h / (n_heads /
 * n_kv_heads), over the kv_len cached positions j,
 *   s_j = scale * sum_d q[h][d] * k[g][j][d]
 *   p_j = exp(s_j - max_j s_j) / sum_j exp(s_j - max_j s_j)
 *   out[h][d] = sum_j p_j * v[g][j][d]
 * with k and v the dequantized cache elements (each rounded once to float,
 * as oracle_dequant gives them), everything else in double. The caches are
 * packed tensors of n_kv_heads * kv_len * head_dim elements, element
 * (g * kv_len + j) * head_dim + d. Also returned per output: A[h][d] =
 * sum_j p_j * |v[g][j][d]|, and per head T[h] = max_j scale * sum_d |q k|. */
int oracle_attn_decode(int fmt, const float* q, const uint8_t* Kc, const uint8_t* Vc, int64_t n_heads,
                       int64_t n_kv_heads, int64_t head_dim, int64_t kv_len, double scale, double* out,
                       double* A, double* T) {
    int64_t offk[4], offv[4], total;
    if (n_heads < 1 || n_kv_heads < 1 || head_dim < 1 || kv_len < 1 || n_heads % n_kv_heads) return -1;
    int64_t n = n_kv_heads * kv_len * head_dim;
    if (planes(fmt, n, offk, &total) || planes(fmt, n, offv, &total) || head_dim % block_elems(fmt)) return -1;
    double* s = (double*)malloc(sizeof(double) * (size_t)kv_len);
    double* t = (double*)malloc(sizeof(double) * (size_t)kv_len);
    if (!s || !t) {
        free(s);
        free(t);
        return -1;
    }
    int64_t group = n_heads / n_kv_heads;
    for (int64_t h = 0; h < n_heads; ++h) {
        int64_t g = h / group;
        const float* qh = q + h * head_dim;
        double smax = -INFINITY, tmax = 0.0;
        for (int64_t j = 0; j < kv_len; ++j) {
            double acc = 0.0, mag = 0.0;
            for (int64_t d = 0; d < head_dim; ++d) {
                double k = (double)(float)exact_value(fmt, Kc, offk, (g * kv_len + j) * head_dim + d);
                acc += (double)qh[d] * k;
                mag += fabs((double)qh[d] * k);
            }
            s[j] = scale * acc;
            t[j] = fabs(scale) * mag;
            if (s[j] > smax) smax = s[j];
            if (t[j] > tmax) tmax = t[j];
        }
        double denom = 0.0;
        for (int64_t j = 0; j < kv_len; ++j) {
            s[j] = exp(s[j] - smax);
            denom += s[j];
        }
        for (int64_t d = 0; d < head_dim; ++d) {
            double o = 0.0, a = 0.0;
            for (int64_t j = 0; j < kv_len; ++j) {
                double v = (double)(float)exact_value(fmt, Vc, offv, (g * kv_len + j) * head_dim + d);
                o += s[j] * v;
                a += s[j] * fabs(v);
            }
            out[h * head_dim + d] = o / denom;
            if (A) A[h * head_dim + d] = a / denom;
        }
        if (T) T[h] = tmax;
    }
    free(s);
    free(t);
    return 0;
}
