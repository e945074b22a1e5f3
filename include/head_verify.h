/*
 * head_verify.h -- C ABI of the output-head candidate-row verification.
 *
 * Operation (paper Sec. 5, "Output-Head Power Case Study", projection-only
 * trace configuration), for the vocabulary projection Q [V][K] (row-major
 * INT8, one FP32 scale per row) and one FP32 activation vector x [K]:
 *
 *  1. x is quantized to INT8 with one scale for the vector, by the Sec. 2.3
 *     formulas: s_x = max(max_k |x_k|, 1e-8) / 127, xq = clip(round(x / s_x),
 *     -127, 127), in binary32 with ties to even;
 *  2. approximate logits: logits[m] = fl32(fl32(acc_m) * fl32(scale[m] * s_x))
 *     with acc_m = sum_k Q[m][k] xq_k exact in INT32;
 *  3. candidates: the top_k rows with the largest approximate logits, largest
 *     first, equal logits in ascending row order;
 *  4. gate: gap = fl32(l(1) - l(2)) over the two largest approximate logits of
 *     all V rows (+inf when V = 1); verification runs when gap < threshold;
 *  5. verification: each candidate's logit with the FP32 activations,
 *     scale[m] * sum_k float(Q[m][k]) x_k, in the order of the dense register
 *     kernel (dense_proj.h), so it is bit for bit dense_proj_forward's output
 *     for row m: per lane an FMA chain over the 16-byte chunks l + 32 j
 *     (at most 16 ceil(K/512) products), a 5-level lane tree, one multiply;
 *     error bound as for dense_proj.h with h = 16 ceil(K/512) + 6.  The
 *     token is the candidate with the largest such logit (ties: lower row).
 *     Without verification the token is the top candidate.
 *
 * Steps 1-3 and the gate decision are exact (bit-identical to the
 * definition); step 5 is FP32 arithmetic within the stated bound.
 *
 * Arguments (DEVICE pointers):
 *   Q            int8  [V][K] row-major, 16-byte aligned, K % 16 == 0,
 *                16 <= K <= 4096, 1 <= V, V * K < 2^31.
 *   scale        float [V].
 *   x            float [K], 4-byte aligned.
 *   top_k        1 <= top_k <= min(64, V).
 *   threshold    gate threshold (not NaN; 0 never verifies, +inf verifies
 *                whenever V >= 2).
 *   logits       float [V] out: the approximate logits of step 2.
 *   cand         int32 [top_k] out: candidate rows, best first.
 *   cand_logits  float [top_k] out: the recomputed logits when verification
 *                ran, else the candidates' approximate logits.
 *   result       int32 [2] out: {token, 1 if verification ran else 0}.
 *   workspace    device memory of head_verify_workspace_bytes() bytes,
 *                16-byte aligned, owned by the caller; no initial contents
 *                are needed and nothing in it outlives the call.  Calls that
 *                share a workspace must not overlap: enqueue them on one
 *                stream, or give each stream its own workspace.
 * Two kernels are enqueued on `stream` (a hipStream_t, NULL for the default
 * stream): the approximate head, which when threshold > 0 also computes
 * every row's FP32-activation logit from the same weight registers and keeps
 * those of its listed rows, and the selection, gate and verification.  The gate is decided on the device, so the call never
 * waits for the GPU and can be captured in a HIP graph.  Nothing is
 * allocated.
 *
 * Errors: SPIKE_OK (0) or a negative code from spike_proj.h, with the
 * message in spike_proj_last_error(); arguments are validated before any
 * HIP call.
 */
#ifndef HEAD_VERIFY_H
#define HEAD_VERIFY_H

#include <stdint.h>

#include "spike_proj.h"

#ifdef __cplusplus
extern "C" {
#endif

#define HEAD_MAX_TOP_K 64
#define HEAD_MAX_K 4096

/* Bytes of the workspace head_verify_forward needs (the same for every V). */
int64_t head_verify_workspace_bytes(void);

int head_verify_forward(const int8_t *Q, const float *scale, int32_t K, int32_t V, const float *x, int32_t top_k,
                        float threshold, float *logits, int32_t *cand, float *cand_logits, int32_t *result,
                        void *workspace, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* HEAD_VERIFY_H */
