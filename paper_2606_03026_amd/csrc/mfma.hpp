// Dense i8 matrix-core contraction over the 0/1 spike matrix, for prefill-
// sized batches (gfx950 v_mfma_i32_16x16x64_i8).
//
// For B spike rows the projection of Eq. (sparse) (paper Sec. 2.3) is the
// integer product acc[b][n] = sum_k x[b][k] * Q[n][k] with x in {0,1}; the
// matrix cores compute it densely (every column is read once per row tile
// instead of once per active (row, column) pair) and it stays exact: every
// product is 0 or a weight, and INT32 sums are exact.  The FP32 epilogue is
// the same single conversion and multiply as the gather path, so both paths
// give identical bits.
//
// Layout.  Weights stay column-major and borrowed (W[k*N + n]); the matrix
// core wants 16 consecutive k of one column n in each lane, so every lane
// loads 4 bytes (4 channels) from each of 16 consecutive k-rows and
// transposes the 16x4 byte block in registers with v_perm: the result is the
// B-operand of four MFMAs, one per channel offset t in 0..3, covering the
// channel sets {n0 + 4c + t : c = 0..15}.  The spike bits of a 64-row tile
// are expanded to 0/1 bytes in LDS (double-buffered) and read as A-operands.
// Output layout of the 16x16 i32 accumulator (checked on the device): lane
// l, register j holds row 4*(l/16) + j, column l%16.
//
// Work split: a workgroup owns 64 rows x (64 * WAVES) channels and a range
// of K (whole 64-bit mask words); K-splits fold into the INT32 workspace with
// atomic adds and the last split of a tile writes the result, exactly as in
// the gather path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spk {

constexpr int kMfmaNAlign = 64;  // N must be a multiple of this; W 4-byte aligned
constexpr int kMfmaRows = 64;    // spike rows per workgroup (4 subtiles of 16)
constexpr int kMfmaK = 64;       // k per step: one mask word
constexpr int kXPitch = 80;      // LDS bytes per expanded row (64 + 16 padding)

typedef int32_t mf_i32x4 __attribute__((ext_vector_type(4)));

inline bool mfma_supported(int K, int N, const void* W)
{
    (void)K;
    return N % kMfmaNAlign == 0 && reinterpret_cast<uintptr_t>(W) % 4 == 0;
}

// Four spike bits -> four bytes holding 0 or 1 (bit i -> byte i).
__device__ inline uint32_t expand_nibble(uint32_t bits) { return ((bits & 0xFu) * 0x00204081u) & 0x01010101u; }

// 4x4 byte transpose: d[j] holds 4 channels of k-row j; e[t] gets the 4
// k-rows of channel t.
__device__ inline void transpose4x4(uint32_t d0, uint32_t d1, uint32_t d2, uint32_t d3, uint32_t& e0, uint32_t& e1,
                                    uint32_t& e2, uint32_t& e3)
{
    const uint32_t lo01 = __builtin_amdgcn_perm(d1, d0, 0x05010400u);  // d0.0 d1.0 d0.1 d1.1
    const uint32_t hi01 = __builtin_amdgcn_perm(d1, d0, 0x07030602u);  // d0.2 d1.2 d0.3 d1.3
    const uint32_t lo23 = __builtin_amdgcn_perm(d3, d2, 0x05010400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(d3, d2, 0x07030602u);
    e0 = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);  // d0.0 d1.0 d2.0 d3.0
    e1 = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    e2 = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    e3 = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

template <int WAVES, bool ACC>
__global__ __launch_bounds__(64 * WAVES) void k_mfma(const int8_t* __restrict__ W, const float* __restrict__ scale,
                                                     int K, int N, const uint64_t* __restrict__ mask, int wpr, int B,
                                                     int words_per_split, int n_splits, int n_coltiles, int32_t* ws,
                                                     uint32_t* counters, float* out, int32_t* acc_out)
{
    constexpr int BLOCK = 64 * WAVES;
    constexpr int COLS = 64 * WAVES;
    __shared__ __align__(16) uint8_t xs[2][kMfmaRows * kXPitch];
    __shared__ int32_t is_last;

    const int wave = threadIdx.x / 64;
    const int l = threadIdx.x % 64;
    const int q = l / 16;  // k-group of the operands, row group of the result
    const int c = l % 16;  // row of A, column of B and of the result
    const int split = blockIdx.x % n_splits;
    const int rest = blockIdx.x / n_splits;
    const int ct = rest % n_coltiles;
    const int rt = rest / n_coltiles;
    const int m0 = rt * kMfmaRows;
    const int n0 = ct * COLS + wave * 64;  // this wave's 64 channels
    const bool wave_on = n0 < N;
    const int w_begin = split * words_per_split;
    const int w_end = min(wpr, w_begin + words_per_split);

    // Stage the spikes of mask word w (64 k) for the tile's 64 rows as 0/1
    // bytes: (row, quarter) pairs spread over the threads.
    auto stage = [&](int buf, int w) {
        for (int p = threadIdx.x; p < kMfmaRows * 4; p += BLOCK) {
            const int r = p >> 2, qq = p & 3;
            const int b = m0 + r;
            uint32_t bits = 0;
            if (b < B && w < w_end) {
                uint64_t word = mask[(int64_t)b * wpr + w];
                const int valid = K - 64 * w;
                if (valid < 64)
                    word &= valid <= 0 ? 0ull : ((1ull << valid) - 1ull);
                bits = (uint32_t)(word >> (16 * qq)) & 0xFFFFu;
            }
            uint4 v;
            v.x = expand_nibble(bits);
            v.y = expand_nibble(bits >> 4);
            v.z = expand_nibble(bits >> 8);
            v.w = expand_nibble(bits >> 12);
            *reinterpret_cast<uint4*>(&xs[buf][r * kXPitch + qq * 16]) = v;
        }
    };
    // 4 channels (n0 + 4c ..) of k-rows kb + 16q + i, i < 16; rows past K are
    // clamped to a valid row (their spikes are zero).
    const int8_t* wbase = W + n0 + 4 * c;
    auto load_w = [&](int kb, uint32_t (&d)[16]) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int k = min(kb + 16 * q + i, K - 1);
            d[i] = *reinterpret_cast<const uint32_t*>(wbase + (int64_t)k * N);
        }
    };

    mf_i32x4 acc[4][4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int t = 0; t < 4; ++t)
            acc[ms][t] = mf_i32x4{0, 0, 0, 0};

    uint32_t wc[16], wn[16];
    if (wave_on && w_begin < w_end)
        load_w(w_begin * kMfmaK, wc);
    stage(0, w_begin);
    __syncthreads();
    int buf = 0;
    for (int w = w_begin; w < w_end; ++w) {
        const bool more = w + 1 < w_end;
        if (wave_on && more)
            load_w((w + 1) * kMfmaK, wn);
        if (wave_on) {
            mf_i32x4 f[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                uint32_t e0, e1, e2, e3;
                transpose4x4(wc[4 * m], wc[4 * m + 1], wc[4 * m + 2], wc[4 * m + 3], e0, e1, e2, e3);
                f[0][m] = (int32_t)e0;
                f[1][m] = (int32_t)e1;
                f[2][m] = (int32_t)e2;
                f[3][m] = (int32_t)e3;
            }
#pragma unroll
            for (int ms = 0; ms < 4; ++ms) {
                const mf_i32x4 a = *reinterpret_cast<const mf_i32x4*>(&xs[buf][(ms * 16 + c) * kXPitch + q * 16]);
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    acc[ms][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, f[t], acc[ms][t], 0, 0, 0);
            }
        }
        if (more)
            stage(buf ^ 1, w + 1);
        __syncthreads();
        buf ^= 1;
        if (more) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
                wc[i] = wn[i];
        }
    }

    if (n_splits == 1) {
        if (!wave_on)
            return;
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int b = m0 + 16 * ms + 4 * q + j;
                    if (b < B) {
                        const int64_t n = n0 + 4 * c + t;
                        if constexpr (ACC) {
                            acc_out[(int64_t)b * N + n] = acc[ms][t][j];
                        } else {
                            const float as_float = (float)acc[ms][t][j];
                            out[(int64_t)b * N + n] = as_float * scale[n];
                        }
                    }
                }
        return;
    }

    // K-split: exact INT32 atomics; the last split of the tile writes it.
    if (wave_on) {
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int b = m0 + 16 * ms + 4 * q + j;
                    if (b < B)
                        atomicAdd(ws + (int64_t)b * N + n0 + 4 * c + t, acc[ms][t][j]);
                }
    }
    __threadfence();
    __syncthreads();
    uint32_t* counter = counters + (int64_t)rt * n_coltiles + ct;
    if (threadIdx.x == 0)
        is_last = atomicAdd(counter, 1u) == (uint32_t)(n_splits - 1);
    __syncthreads();
    if (!is_last)
        return;
    __threadfence();
    const int nbase = ct * COLS;
    for (int e = threadIdx.x; e < kMfmaRows * COLS; e += BLOCK) {
        const int b = m0 + e / COLS;
        const int64_t n = nbase + e % COLS;
        if (b < B && n < N) {
            const int32_t sum = atomicExch(ws + (int64_t)b * N + n, 0);
            if constexpr (ACC) {
                acc_out[(int64_t)b * N + n] = sum;
            } else {
                const float as_float = (float)sum;
                out[(int64_t)b * N + n] = as_float * scale[n];
            }
        }
    }
    if (threadIdx.x == 0)
        atomicExch(counter, 0u);
}

// Launch over B rows: splits of K chosen so that about 512 workgroups run,
// unless words_per_split_req > 0 fixes it.  Needs a workspace of B*N INT32
// and ceil(B/64) * ceil(N/(64*waves)) counters, both zero.
inline hipError_t launch_mfma(const int8_t* W, const float* scale, int K, int N, const uint64_t* mask, int B,
                              int words_per_split_req, int32_t* ws, uint32_t* counters, float* out, int32_t* acc,
                              bool want_acc, hipStream_t st)
{
    const int wpr = (K + 63) / 64;
    const int waves = B <= 64 ? 1 : 4;
    const int cols = 64 * waves;
    const int n_coltiles = (N + cols - 1) / cols;
    const int n_rowtiles = (B + kMfmaRows - 1) / kMfmaRows;
    const int64_t base = (int64_t)n_coltiles * n_rowtiles;
    int wps = words_per_split_req;
    if (wps <= 0) {
        int64_t splits = (512 + base - 1) / base;
        splits = splits < 1 ? 1 : (splits > wpr ? wpr : splits);
        wps = (int)((wpr + splits - 1) / splits);
    }
    wps = wps < 1 ? 1 : (wps > wpr ? wpr : wps);
    const int n_splits = (wpr + wps - 1) / wps;
    const int64_t units = base * n_splits;
    if (units > 0x7fffffff)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)units);
    if (waves == 1) {
        if (want_acc)
            hipLaunchKernelGGL((k_mfma<1, true>), grid, dim3(64), 0, st, W, scale, K, N, mask, wpr, B, wps, n_splits,
                               n_coltiles, ws, counters, out, acc);
        else
            hipLaunchKernelGGL((k_mfma<1, false>), grid, dim3(64), 0, st, W, scale, K, N, mask, wpr, B, wps, n_splits,
                               n_coltiles, ws, counters, out, acc);
    } else {
        if (want_acc)
            hipLaunchKernelGGL((k_mfma<4, true>), grid, dim3(256), 0, st, W, scale, K, N, mask, wpr, B, wps,
                               n_splits, n_coltiles, ws, counters, out, acc);
        else
            hipLaunchKernelGGL((k_mfma<4, false>), grid, dim3(256), 0, st, W, scale, K, N, mask, wpr, B, wps,
                               n_splits, n_coltiles, ws, counters, out, acc);
    }
    return hipGetLastError();
}

}  // namespace spk
