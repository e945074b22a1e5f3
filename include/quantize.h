/*
 * quantize.h -- C ABI of the symmetric per-channel INT8 quantizer and
 * exporter.
 *
 * Operation (paper Sec. 2.3, "Quantization and Accumulation"): for a weight
 * matrix W [M][K] whose row m belongs to output channel m,
 *
 *     scale[m] = max(max_k |W[m][k]|, 1e-8) / 127
 *     Q[m][k]  = clip(round(W[m][k] / scale[m]), -127, 127)
 *
 * in binary32 arithmetic: the maximum is exact, 1e-8 is its nearest binary32
 * value, both divisions are correctly rounded, and round() takes ties to
 * even.  The floor keeps an all-zero row finite (its Q is all zero).
 * Results are bit-identical to that definition.  Non-finite weights give
 * unspecified (but finite, in range) codes.
 *
 * Layouts of Q (all pointers are DEVICE pointers):
 *   SPIKE_LAYOUT_ROW_MAJOR  Q[m*K + k]: the dense continuous-input kernels
 *                           (dense_proj.h).
 *   SPIKE_LAYOUT_COL_MAJOR  Q[k*M + m]: the spike-gated projections
 *                           (spike_proj.h's W, with N = M): the column of
 *                           input k is M contiguous bytes (Sec. 2.2).
 * W is float [M][K] row-major; scale is float [M], one per OUTPUT channel in
 * both layouts.  Scales are always computed along the output axis of the
 * logical [M][K] matrix, before any transposition, so the export defect the
 * paper withdraws (App. "Pure-INT4 Export Correction": scales taken after
 * transposing to [K][M]) cannot arise here.
 *
 * Sizes: 1 <= M, K <= 2^24 and M * K <= 2^31.  The call enqueues two kernels
 * on `stream` (a hipStream_t, NULL for the default stream) and returns; it
 * allocates nothing.  Q and scale must not overlap W.
 *
 * Errors: SPIKE_OK (0) or a negative code from spike_proj.h, with the
 * message in spike_proj_last_error(); arguments are validated before any HIP
 * call.
 */
#ifndef SPIKE_QUANTIZE_H
#define SPIKE_QUANTIZE_H

#include <stdint.h>

#include "spike_proj.h"

#ifdef __cplusplus
extern "C" {
#endif

#define SPIKE_LAYOUT_ROW_MAJOR 0
#define SPIKE_LAYOUT_COL_MAJOR 1

int spike_quantize_int8(const float *W, int32_t M, int32_t K, int32_t layout, int8_t *Q, float *scale,
                        void *stream);

/* Host-only check of a stored scale tensor against its weight: for a logical
 * [M][K] weight quantized per output channel in groups of `group` inputs
 * (group = K: one scale per channel), the scales must have shape
 * [M][ceil(K / group)] (scale_cols = 1 for per-channel scales).  A tensor of
 * shape [K][ceil(M / group)] -- the same element count when M and K trade
 * places -- is reported as scales taken along the wrong axis (after a
 * transposition), the defect the paper withdraws.  Returns SPIKE_OK or
 * SPIKE_EINVAL with the reason in spike_proj_last_error(). */
int spike_check_scale_shape(int32_t M, int32_t K, int32_t group, int32_t scale_rows, int32_t scale_cols);

#ifdef __cplusplus
}
#endif

#endif /* SPIKE_QUANTIZE_H */
