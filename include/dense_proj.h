/*
 * dense_proj.h -- C ABI of the dense continuous-input INT8 projection.
 *
 * Operation (paper Sec. 2.3, end of "Quantization and Accumulation", and
 * the lower path of Fig. "execution"): projections whose inputs are
 * continuous FP32 activations (attention query/key/value/output, feed-
 * forward up, vocabulary head) store INT8 weights row by row with one FP32
 * scale per output channel.  Every weight is converted to FP32, the products
 * with the activations are accumulated in FP32 and the scale is applied
 * once:
 *
 *     y[b][m] = scale[m] * sum_k float(Q[m][k]) * x[b][k]
 *
 * Precision: FP32 fused multiply-adds in a fixed order that depends only on
 * K and on the alignment of Q (each output is the sum of 16 or 32 per-lane
 * FMA chains of at most ceil(K/16) + 15 products, combined by a pairwise
 * tree of at most 5 levels, then one FP32 multiply by scale[m]).  Results
 * are deterministic and do not depend on B, but they are not the exactly
 * rounded value: with u = 2^-24, gamma(n) = n u / (1 - n u) and
 * h = ceil(K/16) + 20,
 *     |y - exact| <= u |exact| + (1 + u) scale[m] gamma(h) sum_k |Q[m][k] x[b][k]|.
 * When every partial sum is an integer below 2^24 in magnitude (integer-
 * valued x), the sum is exact and y is the correctly rounded product.
 *
 * Data layout (all pointers are DEVICE pointers):
 *   Q      int8   [M][K]  row-major: Q[m*K + k]; the row of output m is K
 *                         contiguous bytes (the transpose of the spiking
 *                         projections' column-major layout).
 *   scale  float  [M]     one FP32 scale per output channel.
 *   x      float  [B][K]  row-major activations.
 *   y      float  [B][M]  row-major; every element is written.
 *
 * Sizes: 1 <= K <= DENSE_MAX_K, 1 <= M, M * K < 2^31 bytes, 0 <= B <=
 * DENSE_MAX_B (B = 0 launches nothing).  Pointers must be 4-byte aligned
 * (Q any alignment: 16-byte loads when Q is 16-byte aligned and K % 16 == 0,
 * else 4-byte loads when both allow, else byte loads).  Nothing is allocated
 * or retained: the call only enqueues kernels on `stream` (a hipStream_t,
 * NULL for the default stream), one per group of batch rows (each launch
 * streams all of Q; see the kernels below), and returns without
 * synchronising.  y must not
 * overlap Q, scale or x.
 *
 * Errors: SPIKE_OK (0) or a negative code from spike_proj.h; the message is
 * available from spike_proj_last_error().  Arguments are validated before
 * any HIP call; a launch failure returns SPIKE_EHIP.
 */
#ifndef DENSE_PROJ_H
#define DENSE_PROJ_H

#include <stdint.h>

#include "spike_proj.h"

#ifdef __cplusplus
extern "C" {
#endif

#define DENSE_MAX_K 16128
#define DENSE_MAX_B 65535

int dense_proj_forward(const int8_t *Q, const float *scale, int32_t K, int32_t M, const float *x, int32_t B,
                       float *y, void *stream);

/* Kernels: DENSE_KERNEL_REGISTER keeps each lane's slice of the activations
 * in registers (16-byte aligned Q, K % 16 == 0, K <= 4096, up to 4 batch
 * rows per launch); DENSE_KERNEL_STAGED stages them in LDS (any K, alignment,
 * up to 8 rows per launch).  The choice depends on K and Q's alignment only. */
#define DENSE_KERNEL_STAGED 1
#define DENSE_KERNEL_REGISTER 2

/* Launch shape of the first launch dense_proj_forward makes for (K, M, B)
 * and a Q whose address is a multiple of q_align bytes (1, 2, 4, 8 or 16):
 * kernel, bytes per weight load (16, 4 or 1), batch rows per launch and
 * workgroups.  Host-only; any output pointer may be NULL. */
int dense_proj_plan(int32_t K, int32_t M, int32_t B, int32_t q_align, int32_t *kernel, int32_t *vec,
                    int32_t *rows_per_launch, int32_t *workgroups);

/* Process-wide launch-shape overrides, for measurements; 0 restores the
 * automatic choice.  DENSE_TUNE_KERNEL forces a kernel (the register kernel
 * only where it applies; results differ between the two kernels in the last
 * bits, each within the bound above).  DENSE_TUNE_WG_PER_CU caps the
 * register kernel's grid at value * 256 workgroups (results unchanged). */
#define DENSE_TUNE_KERNEL 1
#define DENSE_TUNE_WG_PER_CU 2
int dense_proj_tune(int32_t key, int32_t value);

#ifdef __cplusplus
}
#endif

#endif /* DENSE_PROJ_H */
