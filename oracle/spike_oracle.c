/*
 * Reference oracle for the spike-gated INT8 projection.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain CPU definition that
 * the GPU library is checked against.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it; the library never calls
 * it and shares no code, header or table with it.
 *
 * What it computes (paper Sec. 2.2 and Sec. 2.3, Eq. (sparse) and the caption
 * of Fig. "execution"):
 *
 *   For a binary input x in {0,1}^K, the active index set is
 *   A = { k : x_k = 1 }.  The quantized weight Q (INT8, one row per output
 *   channel m) is stored column-major, so column k is contiguous across the
 *   output channels.  The projection is  y_m = s_m * sum_{k in A} Q_{m,k}:
 *   the integer weights of the active columns are summed in an INT32
 *   accumulator, and the sum is converted to FP32 and multiplied once by the
 *   per-output-channel FP32 scale s_m.
 *
 * Naming: the paper's output index m is called n here and the number of
 * output channels N; W[k*N + n] = Q_{n,k}.  Spike rows are packed bitmasks:
 * row b holds ceil(K/64) 64-bit words, bit k is bit (k % 64) of word k/64;
 * bits at positions >= K are padding and are ignored.
 *
 * Precision: the paper fixes INT32 accumulation and an FP32 result, so the
 * epilogue is one int->float conversion and one binary32 multiply (no fused
 * multiply-add; the build uses -ffp-contract=off and no fast-math).
 *
 * Domain: 1 <= K <= 2^24 keeps every INT32 sum in range (|Q| <= 128).
 *
 * Pinned by tests/test_oracle_pins.py: brute-force dense integer products,
 * the all-zero / all-one / single-spike special cases, additivity over
 * disjoint spike sets, a hand-worked example (tests/golden), and a
 * numpy float32 re-derivation of the epilogue.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>

#define ORACLE_MAX_K (1LL << 24)

/* Spike bit k of one packed row. */
static int spike_bit(const uint64_t *row, int64_t k)
{
    return (int)((row[k / 64] >> (k % 64)) & 1u);
}

/* Step 1 (Sec. 2.2): the active index set A = {k : x_k = 1}, ascending.
 * Writes |A| indices to idx and returns |A|. */
int64_t oracle_active_indices(const uint64_t *row, int64_t K, int32_t *idx)
{
    int64_t count = 0;
    for (int64_t k = 0; k < K; ++k)
        if (spike_bit(row, k))
            idx[count++] = (int32_t)k;
    return count;
}

/* Step 2 (Eq. (sparse), integer part): for output channels n0 <= n < n1,
 * acc[n - n0] = sum over k in A of Q_{n,k}, read from column k of W. */
static void accumulate_active_columns(const int8_t *W, int64_t N, const int32_t *active,
                                      int64_t n_active, int64_t n0, int64_t n1, int32_t *acc)
{
    for (int64_t n = n0; n < n1; ++n)
        acc[n - n0] = 0;
    for (int64_t a = 0; a < n_active; ++a) {
        const int8_t *column = W + (int64_t)active[a] * N;
        for (int64_t n = n0; n < n1; ++n)
            acc[n - n0] += (int32_t)column[n];
    }
}

/* Step 3 (Sec. 2.3): convert the INT32 sum to FP32, then scale once. */
static float scale_once(int32_t acc, float scale)
{
    float as_float = (float)acc;
    return as_float * scale;
}

static int check_args(const void *W, const void *mask, int64_t K, int64_t N, int64_t B, const void *out)
{
    if (K < 1 || K > ORACLE_MAX_K || N < 1 || B < 0)
        return -1;
    if (B > 0 && (!W || !mask || !out))
        return -1;
    return 0;
}

/* INT32 accumulators for B spike rows: acc[b*N + n]. Returns 0, or -1 on bad
 * arguments. */
int oracle_spike_acc(const int8_t *W, int64_t K, int64_t N, const uint64_t *mask, int64_t B,
                     int32_t *acc)
{
    if (check_args(W, mask, K, N, B, acc))
        return -1;
    const int64_t words = (K + 63) / 64;
    int32_t *active = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
    if (!active)
        return -3;
    for (int64_t b = 0; b < B; ++b) {
        int64_t n_active = oracle_active_indices(mask + b * words, K, active);
        accumulate_active_columns(W, N, active, n_active, 0, N, acc + b * N);
    }
    free(active);
    return 0;
}

struct range_job {
    const int8_t *W;
    const float *scale;
    const uint64_t *mask;
    int64_t K, N, B, words;
    int64_t n0, n1;
    float *out;
    int status;
};

/* One thread's share of oracle_spike_forward: output channels [n0, n1) of
 * every row, each row computed by the three steps above. */
static void *run_range(void *arg)
{
    struct range_job *job = (struct range_job *)arg;
    int64_t width = job->n1 - job->n0;
    int32_t *active = (int32_t *)malloc(sizeof(int32_t) * (size_t)job->K);
    int32_t *acc = (int32_t *)malloc(sizeof(int32_t) * (size_t)(width > 0 ? width : 1));
    if (!active || !acc) {
        free(active);
        free(acc);
        job->status = -3;
        return NULL;
    }
    for (int64_t b = 0; b < job->B; ++b) {
        int64_t n_active = oracle_active_indices(job->mask + b * job->words, job->K, active);
        accumulate_active_columns(job->W, job->N, active, n_active, job->n0, job->n1, acc);
        float *out_row = job->out + b * job->N;
        for (int64_t n = job->n0; n < job->n1; ++n)
            out_row[n] = scale_once(acc[n - job->n0], job->scale[n]);
    }
    free(active);
    free(acc);
    job->status = 0;
    return NULL;
}

/* FP32 outputs for B spike rows: out[b*N + n] = fl32(fl32(acc) * scale[n]).
 * With threads > 1 each thread owns a contiguous range of output channels of
 * every row and walks the same active lists, so the result does not depend
 * on the thread count.  Returns 0, -1 on bad arguments, -3 when memory runs
 * out. */
int oracle_spike_forward(const int8_t *W, const float *scale, int64_t K, int64_t N,
                         const uint64_t *mask, int64_t B, float *out, int threads)
{
    if (check_args(W, mask, K, N, B, out) || (B > 0 && !scale))
        return -1;
    if (B == 0)
        return 0;
    if (threads < 1)
        threads = 1;
    if (threads > N)
        threads = (int)N;
    struct range_job *jobs = (struct range_job *)calloc((size_t)threads, sizeof(struct range_job));
    pthread_t *tids = (pthread_t *)calloc((size_t)threads, sizeof(pthread_t));
    int status = 0;
    if (!jobs || !tids) {
        status = -3;
        goto done;
    }
    for (int t = 0; t < threads; ++t) {
        jobs[t].W = W;
        jobs[t].scale = scale;
        jobs[t].mask = mask;
        jobs[t].K = K;
        jobs[t].N = N;
        jobs[t].B = B;
        jobs[t].words = (K + 63) / 64;
        jobs[t].n0 = N * t / threads;
        jobs[t].n1 = N * (t + 1) / threads;
        jobs[t].out = out;
        jobs[t].status = -3;
    }
    if (threads == 1) {
        run_range(&jobs[0]);
    } else {
        int started = 0;
        for (int t = 0; t < threads; ++t, ++started)
            if (pthread_create(&tids[t], NULL, run_range, &jobs[t]) != 0)
                break;
        for (int t = 0; t < started; ++t)
            pthread_join(tids[t], NULL);
        for (int t = started; t < threads; ++t)
            run_range(&jobs[t]);
    }
    for (int t = 0; t < threads; ++t)
        if (jobs[t].status != 0)
            status = jobs[t].status;
done:
    free(jobs);
    free(tids);
    return status;
}

/*
 * Dense continuous-input projection (paper Sec. 2.3, last sentences of
 * "Quantization and Accumulation"; Fig. "execution", lower path): weights of
 * the continuous-input projections stay row-major, Q[m*K + k] = Q_{m,k}, one
 * scale s_m per output channel.  Each INT8 weight is converted to a real
 * number, multiplied by the FP32 activation x_k, the products of a row are
 * summed, and the row scale is applied once:
 *
 *   y_m = s_m * sum_k Q_{m,k} * x_k
 *
 * The GPU accumulates in FP32 (the paper's precision); this oracle computes
 * the same expression in float64, which is exact up to one rounding per
 * addition at 2^-53, so comparisons use a tolerance derived from the GPU's
 * FP32 summation tree.  x is B rows of K floats, y is B rows of M doubles.
 */
int oracle_dense_forward(const int8_t *Q, const float *scale, int64_t K, int64_t M, const float *x,
                         int64_t B, double *y)
{
    if (K < 1 || M < 1 || B < 0)
        return -1;
    if (B > 0 && (!Q || !scale || !x || !y))
        return -1;
    for (int64_t b = 0; b < B; ++b) {
        const float *xb = x + b * K;
        for (int64_t m = 0; m < M; ++m) {
            const int8_t *row = Q + m * K;
            double dot = 0.0;
            for (int64_t k = 0; k < K; ++k)
                dot += (double)row[k] * (double)xb[k];
            y[b * M + m] = (double)scale[m] * dot;
        }
    }
    return 0;
}
