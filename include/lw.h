/*
 * lw.h — C ABI of the fused dequantize x matrix-vector library for MI355X (gfx950).
 *
 * The operation is the decode step of a transformer run with block-quantized
 * weights: y = dequant(W) . x (paper Sec. 2.1, decode is a matrix-vector
 * product; Sec. 3.3, matrix-vector kernels dequantize weights in registers).
 * The element value of every format follows Eq. (1) of Sec. 2.2,
 * x_hat = s * q + mu, with the block structure of Sec. 2.2 (legacy blocks of
 * 32 weights; K-quant super-blocks of 256 = 8 sub-blocks of 32 whose scales are
 * themselves quantized against a super-block scale).
 *
 * Every entry point is extern "C", takes plain pointers and 64-bit sizes, and
 * needs no HIP or C++ header from the caller. Pointers named "device" must be
 * device (HBM) addresses; the library never dereferences them on the host.
 *
 * Ownership: the caller owns every buffer. The library allocates no memory and
 * keeps no pointer after a call returns. Its only state is immutable, so every
 * entry point is re-entrant and thread-safe.
 *
 * Asynchrony: lw_matvec and lw_dequant only enqueue work and return; they never
 * synchronise. A launch error is reported as LW_EHIP; an error inside a running
 * kernel surfaces on the caller's next synchronisation.
 *
 * Errors: every argument is checked on the host, in the order of the codes
 * below (format, then values, then shape, then alignment), before any HIP call.
 * A call that returns an error has launched nothing and written nothing.
 *
 * ------------------------------------------------------------------------
 * Packed layout ("lw split-plane layout").
 *
 * A tensor of n elements is stored as up to three planes that follow each
 * other from the base pointer W. Plane 0 starts at W; each later plane starts
 * at the end of the previous one rounded up to a multiple of 256 bytes. All
 * multi-byte fields are little-endian; "binary16" is IEEE 754 half precision.
 * Elements are numbered e = 0..n-1; for a matrix of M rows and K columns,
 * e = r*K + k (row-major). Group g = e / 32; super-block S = e / 256; sub-block
 * j = (e / 32) mod 8.
 *
 *   LW_F16  plane 0: n x binary16.                      value = fp16[e]
 *   LW_Q8_0 plane 0: n x int8 (two's complement) q.
 *           plane 1: n/32 x binary16 d.                  value = q[e] * d[g]
 *   LW_Q4_0 plane 0: n/2 bytes; group g owns bytes [16g, 16g+16); byte i of
 *                    the group holds element 32g+i in bits 0-3 and element
 *                    32g+i+16 in bits 4-7 (unsigned codes q in [0, 15]).
 *           plane 1: n/32 x binary16 d.                  value = (q - 8) * d[g]
 *   LW_Q4_K plane 0: as LW_Q4_0 plane 0 (group g = 8S + j).
 *           plane 1: n/256 records of 12 bytes. A record is a 96-bit
 *                    little-endian integer R with sc_j = (R >> 6j) & 63 and
 *                    m_j = (R >> (48 + 6j)) & 63, j = 0..7.
 *           plane 2: n/256 x { binary16 d, binary16 dmin } (4 bytes each).
 *                                    value = d[S] * sc_j * q[e] - dmin[S] * m_j
 *   LW_Q4_1 plane 0: as LW_Q4_0 plane 0.
 *           plane 1: n/32 x { binary16 d, binary16 m } (4 bytes each).
 *                                    value = q[e] * d[g] + m[g]
 *   LW_Q1_0 plane 0: n/8 bytes; element e is bit (e mod 8) of byte e/8
 *                    (code b in {0, 1}, standing for the level 2b - 1).
 *           plane 1: n/128 x binary16 d (block B = e / 128).
 *                                    value = (2b[e] - 1) * d[B] = +-d[B]
 *
 *   5-bit codes q in [0, 31]: bits 0-3 in a plane laid out as LW_Q4_0's plane
 *   0, bit 4 in a plane of n/8 bytes (element e at bit (e mod 8) of byte e/8).
 *   LW_Q5_0 plane 0: low four bits; plane 1: fifth bits;
 *           plane 2: n/32 x binary16 d.            value = (q - 16) * d[g]
 *   LW_Q5_1 planes 0, 1 as LW_Q5_0; plane 2: n/32 x { binary16 d, binary16 m }.
 *                                                   value = q * d[g] + m[g]
 *   LW_Q5_K planes 0, 1 as LW_Q5_0; plane 2: the 12-byte records of LW_Q4_K;
 *           plane 3: n/256 x { binary16 d, binary16 dmin }.
 *                                    value = d[S] * sc_j * q[e] - dmin[S] * m_j
 *   Sub-blocks of 16 (t = e / 16):
 *   LW_Q6_K plane 0: bits 0-3 of 6-bit codes q in [0, 63], as LW_Q4_0's
 *                    plane 0; plane 1: n/4 bytes of bits 4-5, element e at
 *                    bits 2(e mod 4) .. 2(e mod 4)+1 of byte e/4;
 *           plane 2: n/16 x int8 scale sc[t]; plane 3: n/256 x binary16 d.
 *                                    value = d[S] * sc[t] * (q[e] - 32)
 *   LW_Q2_K plane 0: n/4 bytes of 2-bit codes q in [0, 3], element e at bits
 *                    2(e mod 4) .. 2(e mod 4)+1 of byte e/4;
 *           plane 1: n/16 bytes, sc[t] in bits 0-3 and m[t] in bits 4-7;
 *           plane 2: n/256 x { binary16 d, binary16 dmin }.
 *                                    value = d[S] * sc[t] * q[e] - dmin[S] * m[t]
 *   LW_MXFP4 plane 0: 4-bit e2m1 codes as LW_Q4_0's plane 0 (bit 3 the sign,
 *                    bits 1-2 an exponent e with bias 1, bit 0 a mantissa m:
 *                    e2m1 = m/2 for e = 0, else 2^(e-1) * (1 + m/2));
 *           plane 1: n/32 bytes, an e8m0 exponent E per group.
 *                                    value = e2m1(q[e]) * 2^(E[g] - 127)
 *                    (E = 255 is NaN; 2^(E-127) below 2^-126 and products
 *                    beyond binary32's range round as binary32 does)
 *
 * The dequantized value of an element is the exact real value of its closed
 * form rounded once to binary32 with round-to-nearest-even. For LW_F16,
 * LW_Q8_0 and LW_Q4_0 the closed form is exactly representable in binary32;
 * for LW_Q4_K the two products are exact and the difference is rounded once;
 * for LW_Q4_1 the product is exact and the sum with the min is rounded once;
 * LW_Q1_0's value is +-d, exact. LW_Q5_0 and LW_Q6_K are exact; LW_Q5_1,
 * LW_Q5_K and LW_Q2_K round once, as LW_Q4_1 and LW_Q4_K. LW_MXFP4 is exact
 * except for overflow to infinity.
 * ------------------------------------------------------------------------
 */
#ifndef LW_H
#define LW_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The entry points below are the library's only exported symbols (it is
 * built with hidden visibility), so no symbol of a host program can take the
 * place of one of its internal functions. */
#if defined(__GNUC__) || defined(__clang__)
#define LW_API __attribute__((visibility("default")))
#else
#define LW_API
#endif

/* Weight formats (Sec. 2.2: f16 storage, legacy blocks of 32 without (Q8_0,
 * Q4_0, Q5_0) and with (Q4_1, Q5_1) an offset, K-quant super-blocks of 256
 * with double-quantized scales (and mins) at 2, 4, 5 and 6 bits per code,
 * and the 1-bit symmetric q1_0 with one scale per 128 weights; Sec. 7 and
 * Appendix B list q2_k .. q6_k; mxfp4, 4-bit floats with a shared
 * power-of-two scale, which the paper emulates for gpt-oss and MI355X's
 * matrix cores take natively). */
typedef enum {
    LW_F16 = 0, LW_Q8_0 = 1, LW_Q4_0 = 2, LW_Q4_K = 3, LW_Q4_1 = 4, LW_Q1_0 = 5,
    LW_Q5_0 = 6, LW_Q5_1 = 7, LW_Q5_K = 8, LW_Q6_K = 9, LW_Q2_K = 10, LW_MXFP4 = 11
} lw_fmt;

/* Return codes. */
enum {
    LW_OK = 0,
    LW_EINVAL = -1, /* null pointer, or a size out of range (M, K, n_tok < 1; n < 0; too large) */
    LW_EFMT = -2,   /* unknown format */
    LW_ESHAPE = -3, /* K (or n) not a multiple of 256 */
    LW_EALIGN = -4, /* W not 256-byte aligned, or x / y / out not 16-byte aligned */
    LW_EHIP = -5    /* the HIP launch failed */
};

/* Largest accepted M and K, and largest accepted element count M*K or n. */
#define LW_MAX_DIM ((int64_t)1 << 31)
#define LW_MAX_ELEMS ((int64_t)1 << 40)
/* Token blocks of the VALU matrix-vector kernel: f16 and Q8_0 weights take
 * it for up to this many tokens (W streamed once, every token reusing each
 * decoded weight in registers). The 4-bit formats take a VALU kernel for one
 * or two tokens and the matrix cores from three tokens on; Q8_0, Q5_0, Q5_1,
 * Q5_K, Q6_K, Q2_K and MXFP4 take the matrix cores above this bound; f16 and
 * q1_0 stay on the VALU kernel, in token blocks. lw_kernel_name names the
 * kernel a call selects. */
#define LW_GEMV_MAX_TOK 8

/*
 * lw_matvec — y[t][r] = sum_k value(W, r*K + k) * x[t][k]
 *             for 0 <= t < n_tok, 0 <= r < M, 0 <= k < K.
 *
 * Decode step of Sec. 2.1 with the dequantize-in-registers matrix-vector
 * kernel of Sec. 3.3; n_tok > 1 is the multi-token batch of the same product,
 * and n_tok > 16 the prefill matrix multiplication of Sec. 3.2 (dequantized
 * weight tiles reused across tokens, Sec. 3.3).
 *
 *   fmt    one of lw_fmt.
 *   W      device; M*K elements packed in the layout above, 256-byte aligned.
 *   x      device; float32 [n_tok][K] row-major, 16-byte aligned.
 *   y      device; float32 [n_tok][M] row-major, 16-byte aligned; overwritten.
 *          Must not overlap W or x.
 *   M, K   rows and columns; 1 <= M, K <= LW_MAX_DIM, M*K <= LW_MAX_ELEMS;
 *          K must be a multiple of 256 (LW_ESHAPE otherwise).
 *   n_tok  number of token vectors, >= 1.
 *   stream hipStream_t to enqueue on (NULL: the null stream).
 *
 * Arithmetic: products and sums in float32 with float32 accumulation (no
 * reduced-precision activations) on the VALU paths. The matrix-core paths
 * (4-bit formats from three tokens; Q8_0, Q5_0, Q5_1, Q5_K, Q6_K, Q2_K and
 * MXFP4 above LW_GEMV_MAX_TOK tokens) multiply exact bfloat16 codes (integer
 * codes, or the e2m1 values of MXFP4) by activations split into a bfloat16
 * high part and a bfloat16 low part, accumulating in float32. Every path's
 * error relative to sum_k |w * x| stays below 1e-4.
 */
LW_API int lw_matvec(int fmt, const void* W, const float* x, float* y,
              int64_t M, int64_t K, int64_t n_tok, void* stream);

/* Most matrices one lw_matvec_multi call takes. */
#define LW_MULTI_MAX 4

/*
 * lw_matvec_multi — y_i[t][r] = sum_k value(W_i, r*K + k) * x[t][k] for each
 * i < n_mat: several matrices applied to the same activations, the
 * independent projections of one decoder layer (q/k/v, gate/up) in the
 * decode step of Sec. 2.1. Results equal n_mat lw_matvec calls, up to float32
 * summation order. With one token the rows of all matrices form one row space
 * and the call is a single kernel launch (the single-token kernels, selected
 * as for lw_matvec with M = the sum of the M_i). With 3 to 8 tokens (2 to 8
 * for the formats without the two-token register kernel: all but Q4_0, Q4_K,
 * Q4_1 and q1_0) and a format the few-token matrix-core kernel serves (all
 * quantized formats but Q8_0), it is one launch of that kernel where it
 * takes the summed row count (each workgroup then works on rows of one
 * matrix). Otherwise it enqueues one lw_matvec per matrix.
 *
 *   fmt      one of lw_fmt, shared by all matrices.
 *   n_mat    1 <= n_mat <= LW_MULTI_MAX.
 *   W        host array of n_mat device pointers, each as W of lw_matvec.
 *   y        host array of n_mat device pointers, each float32 [n_tok][M[i]],
 *            16-byte aligned, overwritten; no overlap with any W, x or
 *            another y.
 *   M        host array of n_mat row counts, each as M of lw_matvec.
 *   x, K, n_tok, stream  as for lw_matvec, shared by all matrices.
 *
 * Checks as lw_matvec's, in the same order over all matrices (LW_EINVAL also
 * for a null array or n_mat out of range); nothing is launched when one
 * fails. The arrays are read during the call only.
 */
LW_API int lw_matvec_multi(int fmt, int n_mat, const void* const* W, float* const* y, const int64_t* M,
                           const float* x, int64_t K, int64_t n_tok, void* stream);

/*
 * lw_matvec_ws — lw_matvec with a device workspace from the caller, for the
 * paths that need scratch memory. One path does: LW_MXFP4 weights with more
 * than 16 tokens run on MI355X's native fp4 matrix cores (the mxfp4 format of
 * Sec. 2.2 and Appendix B, which the paper emulates): e2m1 codes and their
 * e8m0 exponents go to v_mfma_scale_f32_32x32x64_f8f6f4 as stored. The
 * activations are split once per call into four e2m3 (6-bit float) pieces
 * with one power-of-two scale per 32 values, kept in the workspace; per block,
 * |x - sum of pieces| <= 2^-16 * the block's largest |x|. Error of that path:
 *   |y - exact| <= 2^-16 * sum_k |w_k| * xmax_k + 2^-11 * sum_k |w_k * x_k|,
 * xmax_k the largest |x| of k's 32-block (the second term bounds the matrix
 * core's own summation, which is not float32's). Activations must be finite
 * and below 2^126 in magnitude. Every other call ignores the workspace and
 * is exactly lw_matvec (workspace may then be NULL).
 *
 *   workspace        device, 256-byte aligned, at least
 *                    lw_matvec_workspace_bytes(fmt, M, K, n_tok) bytes, owned
 *                    by the caller; needs no initialisation, undefined
 *                    afterwards. Calls that overlap in time must not share a
 *                    workspace.
 *   workspace_bytes  its size in bytes.
 *   fmt, W, x, y, M, K, n_tok, stream  as for lw_matvec.
 *
 * Checks as lw_matvec's, in the same order; LW_EINVAL also for a workspace
 * that is needed and NULL or too small, LW_EALIGN for one not 256-byte
 * aligned. The fp4 path makes two launches (three where it splits K: each
 * split writes its partial results to the workspace and a last launch sums
 * them into y).
 */
LW_API int lw_matvec_ws(int fmt, const void* W, const float* x, float* y, int64_t M, int64_t K, int64_t n_tok,
                        void* workspace, int64_t workspace_bytes, void* stream);

/*
 * lw_matvec_workspace_bytes — the workspace lw_matvec_ws needs for these
 * sizes (0 where the call takes a path without one; for LW_MXFP4 above 16
 * tokens 100 bytes per 32 activations of n_tok rounded up to 64 tokens, and
 * where the call splits K, 4 bytes per output and split more), or the error
 * lw_matvec would return on format, sizes or shape (negative). Host-only;
 * the same on every device.
 */
LW_API int64_t lw_matvec_workspace_bytes(int fmt, int64_t M, int64_t K, int64_t n_tok);

/*
 * lw_dequant — out[e] = value(W, e) for 0 <= e < n, bit-exact (see above).
 * Runs on the null stream. n == 0 is a no-op returning LW_OK.
 *
 *   W    device; n elements packed in the layout above, 256-byte aligned.
 *   out  device; float32 [n], 16-byte aligned; must not overlap W.
 *   n    element count, 0 <= n <= LW_MAX_ELEMS, a multiple of 256.
 */
LW_API int lw_dequant(int fmt, const void* W, float* out, int64_t n);

/*
 * lw_weight_bytes — size in bytes of n packed elements (plane 0 through the
 * end of the last plane). Returns LW_EFMT, LW_EINVAL (n < 0 or too large) or
 * LW_ESHAPE (n not a multiple of 256) as a negative value. Host-only.
 */
LW_API int64_t lw_weight_bytes(int fmt, int64_t n);

/* lw_strerror — static, NUL-terminated description of a return code. */
LW_API const char* lw_strerror(int code);

/*
 * lw_kernel_name — the kernel lw_matvec(fmt, W, x, y, M, K, n_tok, stream)
 * would launch for these sizes (the first one, where the call launches
 * several), as the template part of its name, e.g. "gemv1r_kernel<3, 1, 2, 1,
 * 8, 2>": the static kernel-selection table of Sec. 3.3 (ahead-of-time
 * instantiations chosen per shape) made visible to profilers and tests.
 *
 *   fmt, M, K, n_tok  as for lw_matvec.
 *
 * Returns NULL when these arguments would fail lw_matvec's checks on format,
 * sizes or shape. The string is owned by the library and valid until the
 * process ends. Host-only: launches nothing and touches no device memory;
 * the selection may depend on the compute-unit count of the current device
 * (256 when there is none).
 */
LW_API const char* lw_kernel_name(int fmt, int64_t M, int64_t K, int64_t n_tok);

/*
 * lw_kernel_name_multi — the kernel lw_matvec_multi(fmt, n_mat, ..., M, x, K,
 * n_tok, stream) would launch: the fused launch's kernel where the call is one
 * launch, else the kernel of its first matrix's lw_matvec. Same string
 * conventions and checks as lw_kernel_name (NULL when the sizes would fail
 * lw_matvec_multi's checks; M is a host array of n_mat row counts).
 * Host-only: launches nothing.
 */
LW_API const char* lw_kernel_name_multi(int fmt, int n_mat, const int64_t* M, int64_t K, int64_t n_tok);

/*
 * lw_kernel_name_ws, lw_launch_count_ws — lw_kernel_name and lw_launch_count
 * for lw_matvec_ws with a large enough workspace. Host-only.
 */
LW_API const char* lw_kernel_name_ws(int fmt, int64_t M, int64_t K, int64_t n_tok);
LW_API int64_t lw_launch_count_ws(int fmt, int64_t M, int64_t K, int64_t n_tok);

/*
 * lw_attn_decode — one query token's attention over a KV cache stored in a
 * weight format, dequantized as it is loaded (Sec. 3.2: attention kernels
 * read quantized K and V; Sec. 3.3: the dequantization routines serve the KV
 * cache as well as the weights). For query head h, its key/value head
 * g = h / (n_heads / n_kv_heads), and the kv_len cached positions j:
 *   s_j = scale * sum_d q[h][d] * k[g][j][d],  p = softmax over j of s,
 *   out[h][d] = sum_j p_j * v[g][j][d].
 *
 *   fmt        LW_F16, LW_Q8_0, LW_Q4_0, LW_Q4_1, LW_Q5_0, LW_Q5_1 or LW_MXFP4
 *              (formats whose blocks fit a head's row); both caches share it.
 *   q          device; float32 [n_heads][head_dim], 16-byte aligned.
 *   K, V       device; each n_kv_heads * kv_len * head_dim elements in the
 *              packed layout above, element (g * kv_len + j) * head_dim + d
 *              (head-major: a head's positions are consecutive rows),
 *              256-byte aligned.
 *   out        device; float32 [n_heads][head_dim], 16-byte aligned,
 *              overwritten; must not overlap the inputs or the workspace.
 *   n_heads, n_kv_heads  n_heads / n_kv_heads in {1, 2, 4, 8}, n_heads <= 4096.
 *   head_dim   64 or 128.   kv_len  1 <= kv_len < 2^31.
 *   scale      finite (usually 1 / sqrt(head_dim)).
 *   workspace  device, 16-byte aligned, at least lw_attn_workspace_bytes(...)
 *              bytes, owned by the caller; holds partial results between the
 *              call's two kernels (its contents need no initialisation and are
 *              undefined afterwards). Calls that overlap in time must not
 *              share a workspace.
 *   stream     hipStream_t (NULL: the null stream).
 *
 * Errors in the usual order: LW_EFMT (fmt not one of the above), LW_EINVAL
 * (null pointer, sizes out of range, a head ratio or head_dim not listed,
 * scale not finite, workspace too small), LW_ESHAPE (n_kv_heads * kv_len *
 * head_dim not a multiple of 256), LW_EALIGN, LW_EHIP. Two kernel launches
 * (lw_attn_kernel_name names the first). Arithmetic in float32, except that
 * f16, Q8_0 and Q4_0 scores on the matrix cores take the query as two f16
 * parts (22 significant bits, after an exact power-of-two scaling per head)
 * times exact f16 forms of the cache elements, with float32 accumulation:
 * each output is within 2^-12 * (1 + T) * sum_j p_j |v[g][j][d]| of the
 * exact value, T the largest scale * sum_d |q k| of the head (the score error
 * enters the weights through exp).
 */
LW_API int lw_attn_decode(int fmt, const float* q, const void* K, const void* V, float* out, int64_t n_heads,
                          int64_t n_kv_heads, int64_t head_dim, int64_t kv_len, float scale, void* workspace,
                          int64_t workspace_bytes, void* stream);

/*
 * lw_attn_workspace_bytes — the workspace lw_attn_decode needs for these
 * sizes (n_heads * splits * (head_dim + 2) * 4 bytes for the library's split
 * of the positions), or the size error of the call (negative). Host-only.
 */
LW_API int64_t lw_attn_workspace_bytes(int fmt, int64_t n_heads, int64_t n_kv_heads, int64_t head_dim,
                                       int64_t kv_len);

/*
 * lw_attn_kernel_name — the first of the two kernels lw_attn_decode launches
 * for these sizes, as "attn_mf_kernel<fmt, head_dim, G>" (f16, Q8_0 and Q4_0
 * caches when the library's split gives more than 64 positions per
 * workgroup: scores on the matrix cores) or "attn_split_kernel<...>" (the
 * vector kernel), G = n_heads / n_kv_heads; NULL when the sizes fail
 * lw_attn_decode's checks. Host-only; the string is static.
 */
LW_API const char* lw_attn_kernel_name(int fmt, int64_t n_heads, int64_t n_kv_heads, int64_t head_dim,
                                       int64_t kv_len);

/*
 * lw_attn_decode_noalloc — lw_attn_decode without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation). It allocates
 * nothing: the partial results go to a fixed 2 MiB array of the library's
 * own on each GPU (held until the process ends), so calls whose
 * lw_attn_workspace_bytes exceeds 2 MiB return LW_EINVAL (32 heads over 8
 * key/value heads of 128 need about 0.5 MiB at any length). Every call on a
 * GPU shares that GPU's array: calls that overlap in time on one GPU race.
 * Arguments, checks and results otherwise as lw_attn_decode's.
 */
LW_API int lw_attn_decode_noalloc(int fmt, const float* q, const void* K, const void* V, float* out,
                                  int64_t n_heads, int64_t n_kv_heads, int64_t head_dim, int64_t kv_len,
                                  float scale, void* stream);

/*
 * lw_launch_count — the number of kernel launches lw_matvec(fmt, W, x, y, M,
 * K, n_tok, stream) makes for these sizes (1 for most calls; 2 where a fill
 * kernel zeroes y before a K-split prefill launch, or where tokens run as
 * two batches). A caller that captures calls into a HIP graph can budget
 * the graph's nodes with it. Returns the count (>= 1), or the error lw_matvec
 * would return on format, sizes or shape (LW_EFMT, LW_EINVAL, LW_ESHAPE).
 * Host-only: launches nothing.
 */
LW_API int64_t lw_launch_count(int fmt, int64_t M, int64_t K, int64_t n_tok);

/*
 * lw_launch_count_multi — the same for lw_matvec_multi(fmt, n_mat, ..., M, x,
 * K, n_tok, stream) (M a host array of n_mat row counts); errors as
 * lw_matvec_multi's size checks (LW_EINVAL also for a null array or n_mat out
 * of range). Host-only.
 */
LW_API int64_t lw_launch_count_multi(int fmt, int n_mat, const int64_t* M, int64_t K, int64_t n_tok);

#ifdef __cplusplus
}
#endif

#endif /* LW_H */
