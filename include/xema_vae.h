/*
 * xema_vae.h -- C ABI of the VAE decoder's upsampling stage, fused.
 *
 * The VAE decoder maps the final latent back to pixels once per request and
 * works close to the output resolution, so its upsampling creates large
 * short-lived activation peaks (Sec. 2.1).  The paper fuses the operators
 * around VAE upsampling, at locations and chunk sizes its plan chooses, to
 * keep such peaks inside the memory budget (Sec. 5.2, "Localized chunking and
 * fusion"; Sec. 8, memory mitigation primitives).  The stage here is nearest
 * 2x upsampling followed by a 3x3 convolution with zero padding 1 and a bias:
 *
 *   U[f, u, v, c] = x[f, u / 2, v / 2, c]                 (integer division)
 *   y[f, u, v, o] = bias[o] + sum over dy, dx in {-1, 0, 1} and c of
 *                   w[o, dy + 1, dx + 1, c] * U[f, u + dy, v + dx, c]
 *
 * with U zero outside the 2H x 2W image.  The fused kernel computes y from x
 * directly: the upsampled image U (as large as y) is never stored, and each
 * output phase (parity of u and v) is a 2x2 convolution of x with weights
 * summed over the 3x3 taps that land on the same source pixel.  Each summed
 * weight is kept as two bf16 values, hi + lo, both applied: 32/36 of the
 * convolution's multiply-adds.  A call may cover a band of source rows, so a
 * caller can produce the output in row bands (chunking); the bytes of every
 * band equal those of the whole-image call.
 *
 * Layout: NHWC (channels last), bfloat16 activations and weights, fp32
 * accumulation, one bf16 rounding of each output.  The summed weights are
 * formed in fp32 and split into hi = bf16(sum) and lo = bf16(sum - hi)
 * (xema_vae_upconv_prepare), which carry each to about 2^-17 of its size,
 * so the output rounding is the only departure from the exact definition
 * beyond fp32 accumulation.
 *
 * Conventions of xema.h apply: status codes, validation before any launch,
 * no device allocation, asynchronous on `stream`, 16-byte device pointers.
 */
#ifndef XEMA_VAE_H_
#define XEMA_VAE_H_

#include <stdint.h>

#include "xema.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Bytes of the phase-summed weights: 4 phases x co x 8 (4 taps, hi then
 * lo) x ci bf16 (64 ci co).  Errors: INVALID_ARG for NULL or non-positive sizes;
 * UNSUPPORTED unless ci is a multiple of 64 and co a multiple of 256.      */
XEMA_API int xema_vae_upconv_weight_bytes(int32_t ci, int32_t co, int64_t* bytes);

/* Forms the phase-summed weights once per layer, asynchronous on `stream`.
 *   w    device, bf16 [co, 3, 3, ci] (OHWI), read only
 *   wp   device, xema_vae_upconv_weight_bytes bytes, written; must not
 *        overlap w
 * With s = the fp32 sum of w[o][ky][kx][c] over the kernel rows ky landing
 * on source row offset a ({0} | {1, 2} when py = 0, {0, 1} | {2} when
 * py = 1) and the columns kx landing on b (the same with px), for output
 * phase p = 2 py + px and source offset t = 2 a + b: wp[p][o][t][c] =
 * bf16(s) and wp[p][o][4 + t][c] = bf16(s - bf16(s)), round to nearest even.
 * Errors: as xema_vae_upconv_weight_bytes; MISALIGNED.                    */
XEMA_API int xema_vae_upconv_prepare(const void* w, int32_t ci, int32_t co, void* wp, void* stream);

/* The upsampling stage over source rows [row_begin, row_begin + row_count)
 * of every frame, i.e. output rows [2 row_begin, 2 (row_begin + row_count)).
 *   x     device, bf16 [n, h, w, ci] (all rows: the band reads its
 *         neighbours), read only; n * h * w * ci * 2 < 2^31
 *   wp    device, from xema_vae_upconv_prepare
 *   bias  device, bf16 [co]
 *   y     device, bf16 [n, 2h, 2w, co]; only the band's rows are written;
 *         must not overlap x, wp or bias
 * Errors (before any launch): INVALID_ARG (NULL, non-positive sizes, a row
 * range outside [0, h), aliasing), UNSUPPORTED (channel multiples as above,
 * input of 2^31 bytes or more), MISALIGNED; XEMA_ERR_HIP if a launch fails. */
XEMA_API int xema_vae_upconv(const void* x, int32_t n, int32_t h, int32_t w, int32_t ci,
                             const void* wp, const void* bias, int32_t co, int32_t row_begin,
                             int32_t row_count, void* y, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* XEMA_VAE_H_ */
