/*
 * spike_proj.h -- C ABI of the MI355X spike-gated INT8 projection library.
 *
 * Operation (paper Sec. 2.2 and Sec. 2.3, Eq. (sparse)):
 *
 *     y[b][n] = scale[n] * sum_{k : x_b[k] = 1} Q[n][k]
 *
 * for binary spike rows x_b in {0,1}^K and INT8 weights Q with N output
 * channels.  The sum over the active columns is exact in INT32; it is then
 * converted to FP32 and multiplied once, in binary32 with round-to-nearest-
 * even and no fused multiply-add, by the per-output-channel FP32 scale.
 * Results are bit-identical to that definition for every launch
 * configuration (integer addition is associative, so the order in which
 * workgroups combine partial sums cannot change them).
 *
 * Data layout (all pointers are DEVICE pointers unless stated):
 *   W      int8   [K][N]  column-major weights: W[k*N + n] = Q[n][k], so the
 *                         column of input k is N contiguous bytes (Sec. 2.2).
 *   scale  float  [N]     one FP32 scale per OUTPUT channel (Sec. 2.3).
 *   mask   uint64 [B][ceil(K/64)]  spike bitmask; bit k of row b is bit
 *                         (k % 64) of little-endian word (k / 64) of that row
 *                         (byte-identical to numpy packbits(bitorder=
 *                         "little") padded to 8-byte rows).  Bits at
 *                         positions >= K are padding and are ignored.
 *   out    float  [B][N]  row-major; every element is written.
 *
 * Ownership: create() BORROWS W and scale (the caller keeps them alive and
 * unchanged until destroy()).  The handle owns a small INT32 workspace of
 * max_B * N entries plus completion counters; the kernels leave it zeroed
 * after every call, so forward() performs no allocation, memset or host
 * synchronisation and can be captured into a HIP graph.  When N % 16 == 0
 * the handle also owns a copy of W in the matrix cores' operand order
 * (ceil(K/64) * 64 * N bytes, made by create() and kept while the reserved
 * batch is at least the matrix-core minimum; the matrix-core path reads
 * only that copy, so W must not change after it is made).  A handle must
 * not run on two streams at the same time (its workspace is shared).
 *
 * Errors: every entry point returns SPIKE_OK (0) or a negative code;
 * spike_proj_last_error() returns a message for the calling thread's last
 * failure.  Arguments are validated before any HIP call.  No C++ exception
 * crosses this interface.  Launch failures are reported as SPIKE_EHIP.
 */
#ifndef SPIKE_PROJ_H
#define SPIKE_PROJ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPIKE_OK 0
#define SPIKE_EINVAL (-1)       /* bad argument (null pointer, size out of range) */
#define SPIKE_EHIP (-2)         /* a HIP runtime call or kernel launch failed */
#define SPIKE_ENOMEM (-3)       /* device or host allocation failed */
#define SPIKE_EUNSUPPORTED (-4) /* valid request this library does not serve */

#define SPIKE_MAX_K (1 << 24) /* keeps every INT32 sum exact: 128 * 2^24 = 2^31 */
#define SPIKE_MAX_N (1 << 24)
#define SPIKE_DEFAULT_MAX_B 512

typedef struct spike_proj *spike_proj_t;
typedef struct spike_stream *spike_stream_t;

/* Create a projection over borrowed column-major INT8 weights W [K][N] and
 * FP32 scales [N] (Sec. 2.2: binary-input projections are stored
 * column-major; Sec. 2.3: one scale per output channel).  1 <= K <=
 * SPIKE_MAX_K, 1 <= N <= SPIKE_MAX_N.  Reserves a workspace for
 * SPIKE_DEFAULT_MAX_B rows on the current device and, when N % 16 == 0 and
 * the copy stays below 2^31 bytes, packs the matrix-core copy of W
 * (synchronous: it waits for the device before and after; if that memory
 * cannot be allocated the handle simply has no matrix-core path).  On
 * success *out_handle is set; on failure it is set to NULL. */
int spike_proj_create(const int8_t *W_int8_colmajor, const float *scale_fp32, int32_t K, int32_t N,
                      spike_proj_t *out_handle);

/* spike_proj_create with the workspace sized for max_B rows (1 <= max_B <=
 * 65535) instead of SPIKE_DEFAULT_MAX_B.  flags: 0, or
 * SPIKE_CREATE_GATHER_ONLY for a handle that never holds the matrix-core
 * copy of W (every call then runs the active-column gather, and the handle
 * holds only a workspace of max_B * N INT32 entries: handles meant for
 * streams of batch-1 projections, or many address-distinct copies of
 * weights).  Unknown flags: SPIKE_EINVAL. */
#define SPIKE_CREATE_GATHER_ONLY 1
int spike_proj_create_reserved(const int8_t *W_int8_colmajor, const float *scale_fp32, int32_t K, int32_t N,
                               int32_t max_B, int32_t flags, spike_proj_t *out_handle);

/* Resize the workspace so that forward() accepts up to max_B rows
 * (1 <= max_B <= 65535).  A max_B below the matrix-core minimum batch
 * (SPIKE_TUNE_MFMA_MIN_B, default 1) also frees the matrix-core copy of W;
 * a max_B at or above it makes the copy again where the shape allows it
 * (never for a SPIKE_CREATE_GATHER_ONLY handle).  Allocates and
 * synchronises the device; call it outside graph capture and while no
 * forward() of this handle is in flight. */
int spike_proj_reserve(spike_proj_t h, int32_t max_B);

/* y = Eq. (sparse) for B spike rows: out[b*N + n].  Asynchronous on
 * `stream` (a hipStream_t; NULL means the default stream).  B = 0 is a
 * no-op; 0 <= B <= the reserved max_B.  Dispatches to the dense i8
 * matrix-core contraction over the 0/1 spike matrix (every product is 0 or
 * a weight, so the sum is the same active-column sum) wherever the handle
 * has the matrix-core copy of W and a matrix-core launch plan can run, from
 * SPIKE_TUNE_MFMA_MIN_B rows (default 1: measured faster than the gather
 * per call at every batch up to 64 and every spike rate from 0.02 to 0.40
 * on the 1536- and 6144-input shapes, since one call is latency-bound);
 * otherwise to the active-column gather.  Both give identical bits.  With
 * SPIKE_PATH_MFMA forced where the matrix-core plan cannot run (no copy of
 * W, a tuned plan that is not instantiated or does not fit, more rows than
 * 31-bit offsets into the mask can address) it returns SPIKE_EUNSUPPORTED. */
int spike_proj_forward(spike_proj_t h, const uint64_t *spike_bitmask, int32_t B, float *out_fp32,
                       void *stream);

/* Same as spike_proj_forward but writes the raw INT32 sums
 * acc[b*N + n] = sum_{k in A_b} Q[n][k] (the accumulator of Sec. 2.3)
 * instead of the scaled FP32 outputs.  Used to check the integer path. */
int spike_proj_forward_acc(spike_proj_t h, const uint64_t *spike_bitmask, int32_t B, int32_t *acc_i32,
                           void *stream);

/* Handle-free variant of spike_proj_forward for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  W and scale are the device arrays that
 * spike_proj_create takes (same layout, borrowed for the call); the result is
 * bit-identical to spike_proj_forward on a handle over them.  The call is
 * served by the active-column gather.  Where that gather splits K across
 * workgroups, its INT32 partial sums and completion counters live in one
 * library-owned device array of SPIKE_STATIC_SCRATCH_WORDS 32-bit words per
 * GPU (4 MiB, held until the process ends), so the call needs
 * B * (N + ceil(N/32)) <= SPIKE_STATIC_SCRATCH_WORDS and returns SPIKE_EINVAL
 * beyond that.  It allocates nothing (no hipMalloc, hipFree or allocating
 * library routine).  Every call on a GPU shares that GPU's array and the
 * kernels leave it zeroed, so calls ordered on one stream are safe but calls
 * that overlap in time on one GPU (two streams, two host threads) race and
 * give wrong results.  Until one call has run outside graph capture on a
 * device, each call also enqueues one small kernel on `stream` that clears
 * the array. */
#define SPIKE_STATIC_SCRATCH_WORDS (1 << 20)
int spike_proj_forward_noalloc(const int8_t *W_int8_colmajor, const float *scale_fp32, int32_t K, int32_t N,
                               const uint64_t *spike_bitmask, int32_t B, float *out_fp32, void *stream);

/* Release the workspace and the handle (waits for the device first).
 * NULL is accepted. */
int spike_proj_destroy(spike_proj_t h);

/* Kernel-path and launch-shape controls, for measurement.  The result never
 * depends on them.  Keys:
 *   SPIKE_TUNE_PATH         SPIKE_PATH_AUTO (default), _GATHER or _MFMA
 *   SPIKE_TUNE_SLICE_WORDS  64-bit mask words per K-slice of the gather
 *                           (0 = automatic; 1..256)
 *   SPIKE_TUNE_MFMA_MIN_B   smallest B sent to the matrix-core path by AUTO
 *                           (default 1)
 *   SPIKE_TUNE_VEC          bytes per lane per column load of the gather:
 *                           0 = automatic, 1, 4, 8 or 16 (16, 8 and 4 need
 *                           N and the W address to be multiples of it)
 *   SPIKE_TUNE_MAX_SLICES   cap on K-slices chosen automatically (1..4096)
 *   SPIKE_TUNE_SHAPE        full gather launch shape, SPIKE_SHAPE(V, LG, U,
 *                           BLOCK): V bytes per lane per column, LG lanes per
 *                           column group, U columns in flight per group,
 *                           BLOCK threads per workgroup; 0 = automatic.  Only
 *                           the shapes the library instantiates are accepted.
 *   SPIKE_TUNE_TILES_PER_UNIT  output-channel tiles handled by one workgroup
 *                           (1..4096); the active list is built once per unit
 *   SPIKE_TUNE_XCD_SPREAD   streams only: 1 = plain unit order; 8 (default) =
 *                           XCD x (workgroups b with b % 8 == x) runs the
 *                           x-th contiguous eighth of the units, so every
 *                           XCD gets the same mix of projections
 *   SPIKE_TUNE_MFMA_WAVES   waves per workgroup of the matrix-core path, which
 *                           share one tile's K range: 0 = automatic, 4, 8, 16
 *   SPIKE_TUNE_MFMA_DEPTH   k-steps of weights in flight per wave of the
 *                           matrix-core path: 0 = automatic, 2, 3, 4, 6, 8, 12 (when a
 *                           wave has at most that many k-steps, all of its
 *                           loads are issued at once)
 *   SPIKE_TUNE_MFMA_ROW_TILE  16-row subtiles per matrix-core workgroup:
 *                           0 = automatic, 1, 2, 4, 8
 *   SPIKE_TUNE_MFMA_COL_SETS  16-channel sets per matrix-core workgroup:
 *                           0 = automatic, 1, 2, 3, 4, 6
 *                           Only the matrix-core plans the library
 *                           instantiates run; forcing SPIKE_PATH_MFMA with
 *                           another combination makes forward() return
 *                           SPIKE_EUNSUPPORTED (AUTO falls back to the
 *                           gather).
 * Returns SPIKE_EINVAL for an unknown key or a value out of range.
 */
#define SPIKE_TUNE_PATH 1
#define SPIKE_TUNE_SLICE_WORDS 2
#define SPIKE_TUNE_MFMA_MIN_B 3
#define SPIKE_TUNE_VEC 4
#define SPIKE_TUNE_MAX_SLICES 5
#define SPIKE_TUNE_SHAPE 6
#define SPIKE_TUNE_TILES_PER_UNIT 7
#define SPIKE_TUNE_XCD_SPREAD 8
#define SPIKE_TUNE_MFMA_WAVES 9
#define SPIKE_TUNE_MFMA_DEPTH 11
#define SPIKE_TUNE_MFMA_ROW_TILE 12
#define SPIKE_TUNE_MFMA_COL_SETS 13
#define SPIKE_SHAPE(V, LG, U, BLOCK) ((V) | ((LG) << 5) | ((U) << 15) | (((BLOCK) / 64) << 20))
#define SPIKE_SHAPE_NT (1 << 25) /* or-ed into a shape code: nontemporal weight loads */
/* or-ed into a shape code: exact 16-bit partial sums (paper Sec. 2.3: bounded
 * active counts may sum in fewer bits); two channels per register, folded
 * into INT32 every 256 columns; results are identical */
#define SPIKE_SHAPE_I16 (1 << 26)
#define SPIKE_PATH_AUTO 0
#define SPIKE_PATH_GATHER 1
#define SPIKE_PATH_MFMA 2
int spike_proj_tune(spike_proj_t h, int32_t key, int32_t value);

/* The launch-shape codes this build instantiates: writes up to `cap` codes
 * to `codes` (host memory; may be NULL when cap is 0) and returns how many
 * exist. */
int spike_proj_shapes(int32_t *codes, int32_t cap);

/* The matrix-core plans this build instantiates, as codes
 * rt | cs << 4 | kw << 8 | d << 16 | preload << 24 | direct << 25 (16-row
 * subtiles and 16-channel sets per workgroup, waves, k-steps of weights in
 * flight per wave, all loads issued at once, spike words loaded with each
 * k-step instead of staged in LDS; the automatic plan of batches up to 4
 * rows is direct): writes up to `cap` codes to `codes` (host memory; may be
 * NULL when cap is 0) and returns how many exist. */
int spike_mfma_plans(int32_t *codes, int32_t cap);

/* Which path a forward() of B rows takes on a handle created for a K x N
 * projection with default tuning and enough reserved rows (assuming the
 * matrix-core copy of W could be allocated): *path receives
 * SPIKE_PATH_GATHER or SPIKE_PATH_MFMA, *plan the matrix-core plan code (as
 * in spike_mfma_plans) or 0.  Host-only: no device is touched. */
int spike_proj_plan_query(int32_t K, int32_t N, int32_t B, int32_t *path, int32_t *plan);

/* Active-index extraction (Sec. 2.2, A = {k : x_k = 1}) as a standalone
 * kernel.  For each row b < B writes the ascending active indices to
 * active_idx[b*K + i], i < active_count[b]; entries past the count are left
 * untouched.  active_idx is int32 [B][K], active_count is int32 [B]. */
int spike_compact(const uint64_t *spike_bitmask, int32_t B, int32_t K, int32_t *active_idx,
                  int32_t *active_count, void *stream);

/* Layer-stack driver (Sec. 2.1: a block runs its TCAM projection and then
 * its FFN down projection; 22 blocks in order).  Runs projs[0..n_proj) in
 * order on `stream`, each on B rows.  Spike masks and outputs are packed per
 * projection, in order: projection j reads B rows of ceil(K_j/64) words
 * starting at word offset sum_{i<j} B*ceil(K_i/64) of `masks`, and writes
 * B*N_j floats starting at sum_{i<j} B*N_i of `out`. */
int spike_stack_forward(const spike_proj_t *projs, int32_t n_proj, const uint64_t *masks, int32_t B,
                        float *out, void *stream);

/* The projections of spike_stack_forward (same arguments, same mask and
 * output layout) in ONE launch on the matrix cores, for callers whose spike
 * inputs are all given up front: no projection's input may depend on an
 * earlier projection's output in the same call (Sec. 2.1: a block's TCAM and
 * down projections, 22 blocks).  One launch instead of n_proj removes the
 * per-launch latency that dominates batched decode (a 1536 x 1536 projection
 * at B = 64 reads 2.4 MB, well under a microsecond at HBM rate).  Requires,
 * for every handle: the same N (a multiple of 16), a matrix-core copy of W
 * (a reserved batch of at least the matrix-core minimum), B rows reserved;
 * at most 64 projections.  Returns SPIKE_EUNSUPPORTED where these do not
 * hold (spike_stack_forward then serves the call).  Results are identical
 * to spike_stack_forward's. */
int spike_stack_forward_fused(const spike_proj_t *projs, int32_t n_proj, const uint64_t *masks, int32_t B,
                              float *out, void *stream);

/* Throughput mode for many independent batch-1 projections: n_tokens
 * tokens, each running n_proj projections, all in one launch.  projs holds
 * n_sets * n_proj handles; token t uses projs[(t % n_sets) * n_proj + j]
 * (n_sets > 1 rotates address-distinct weight copies).  All handles must
 * share N; 1 <= n_proj <= 64 and every K <= 16384.  Per token, masks hold the projections' rows back to back
 * (token stride sum_j ceil(K_j/64) words) and out holds n_proj * N floats.
 * create() copies a small descriptor table to the device (allocates);
 * forward() only launches. */
int spike_stream_create(const spike_proj_t *projs, int32_t n_proj, int32_t n_sets, int32_t n_tokens,
                        spike_stream_t *out_stream);
int spike_stream_forward(spike_stream_t s, const uint64_t *masks, float *out, void *stream);
/* Launch-shape controls of a stream (SPIKE_TUNE_SHAPE, SPIKE_TUNE_TILES_PER_UNIT
 * as for spike_proj_tune); results never depend on them. */
int spike_stream_tune(spike_stream_t s, int32_t key, int32_t value);
int spike_stream_destroy(spike_stream_t s);

/* Message describing the calling thread's most recent failure ("" if none). */
const char *spike_proj_last_error(void);

/* ABI version of this header. */
#define SPIKE_PROJ_ABI_VERSION 2
int spike_proj_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPIKE_PROJ_H */
