/*
 * lw_ceiling.h -- streaming ceilings of the GPU, a measurement aid beside
 * liblw.so (library libceiling.so, built with it).
 *
 * The matrix-vector product and the dequantization are bound by HBM
 * bandwidth. To state how close they come, the benchmark times these two
 * trivial kernels in the same process: the rate a plain 128-bit streaming
 * read (or write) reaches is the practical ceiling for a kernel that moves
 * the same bytes. Neither is part of the product path.
 *
 * Both calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 * stream) and return 0, -1 for invalid arguments (nothing launched) or -5
 * when the launch fails. The caller owns every buffer.
 */
#ifndef LW_CEILING_H
#define LW_CEILING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define LWC_API __attribute__((visibility("default")))
#else
#define LWC_API
#endif

/*
 * lw_ceiling_read -- reads bytes [0, bytes) of the device buffer p with
 * 16-byte non-temporal loads (four in flight per thread, one 512-thread
 * workgroup per compute unit) and folds them into a value that
 * is written to the device word *sink only in the (practically impossible)
 * case that it equals a fixed constant, so the loads cannot be dropped.
 *   p      device, 16-byte aligned.
 *   bytes  a positive multiple of 16.
 *   sink   device uint32_t.
 */
LWC_API int lw_ceiling_read(const void* p, int64_t bytes, uint32_t* sink, void* stream);

/*
 * lw_ceiling_write -- writes zeros over bytes [0, bytes) of the device buffer
 * p with 16-byte non-temporal stores (the dequantization's store form).
 *   p      device, 16-byte aligned.
 *   bytes  a positive multiple of 16.
 */
LWC_API int lw_ceiling_write(void* p, int64_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LW_CEILING_H */
