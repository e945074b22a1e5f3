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
// channel sets {n0 + 4c + t : c = 0..15}.  The spike bits of the tile's 64
// rows are expanded to 0/1 bytes in a per-wave LDS area and read back as
// A-operands.  Output layout of the 16x16 i32 accumulator (checked on the
// device): lane l, register j holds row 4*(l/16) + j, column l%16.
//
// Work split.  A workgroup owns one 64-row x 64-channel tile; its KW waves
// take interleaved 64-wide k-steps of the workgroup's K range and add their
// partial tiles in LDS (LDS atomics).  For small B, K is also split across
// workgroups: each stores its partial tile with plain stores and the last to
// arrive (one counter atomic per workgroup) adds them -- device-scope
// atomics on every output were measured far too slow on this chip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gather.hpp"  // wait_writes_done

namespace spk {

constexpr int kMfmaNAlign = 64;  // N must be a multiple of this; W 4-byte aligned
constexpr int kMfmaRows = 64;    // spike rows per tile (4 subtiles of 16)
constexpr int kMfmaCols = 64;    // channels per tile (4 MFMA channel sets of 16)
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

template <int KW, bool ACC>
__global__ __launch_bounds__(64 * KW) void k_mfma(const int8_t* __restrict__ W, const float* __restrict__ scale,
                                                  int K, int N, const uint64_t* __restrict__ mask, int wpr, int B,
                                                  int words_per_split, int n_splits, int n_coltiles,
                                                  int32_t* __restrict__ parts, uint32_t* counters, float* out,
                                                  int32_t* acc_out)
{
    constexpr int BLOCK = 64 * KW;
    constexpr int TILE = kMfmaRows * kMfmaCols;
    __shared__ __align__(16) uint8_t xs[KW][kMfmaRows * kXPitch];  // one area per wave
    __shared__ int32_t red[TILE];                                  // the tile's INT32 sums
    __shared__ int32_t is_last;

    const int wave = threadIdx.x / 64;
    const int l = threadIdx.x % 64;
    const int q = l / 16;  // k-group of the operands, row group of the result
    const int c = l % 16;  // row of A, column of B and of the result
    const int split = blockIdx.x % n_splits;
    const int tile_id = blockIdx.x / n_splits;
    const int ct = tile_id % n_coltiles;
    const int rt = tile_id / n_coltiles;
    const int m0 = rt * kMfmaRows;
    const int n0 = ct * kMfmaCols;
    const int w_begin = split * words_per_split;
    const int w_end = min(wpr, w_begin + words_per_split);

    for (int e = threadIdx.x; e < TILE; e += BLOCK)
        red[e] = 0;

    uint8_t* xw = xs[wave];
    const int8_t* wbase = W + n0 + 4 * c;
    const int xb = m0 + l;  // the row this lane stages
    // W: 4 channels (n0 + 4c ..) of k-rows kb + 16q + i, i < 16 (rows past K
    // are clamped to a valid row; their spikes are zero).
    auto load_w = [&](int w, uint32_t (&d)[16]) {
        const int kb = w * kMfmaK;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int k = min(kb + 16 * q + i, K - 1);
            d[i] = *reinterpret_cast<const uint32_t*>(wbase + (int64_t)k * N);
        }
    };
    auto load_bits = [&](int w) -> uint64_t {
        if (xb >= B)
            return 0;
        uint64_t word = mask[(int64_t)xb * wpr + w];
        const int valid = K - 64 * w;
        if (valid < 64)
            word &= valid <= 0 ? 0ull : ((1ull << valid) - 1ull);
        return word;
    };
    // this lane's row of the wave's LDS area <- 64 spikes as 0/1 bytes
    auto stage = [&](uint64_t word) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const uint32_t bits = (uint32_t)(word >> (16 * qq));
            uint4 v;
            v.x = expand_nibble(bits);
            v.y = expand_nibble(bits >> 4);
            v.z = expand_nibble(bits >> 8);
            v.w = expand_nibble(bits >> 12);
            *reinterpret_cast<uint4*>(&xw[l * kXPitch + qq * 16]) = v;
        }
    };

    mf_i32x4 acc[4][4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int t = 0; t < 4; ++t)
            acc[ms][t] = mf_i32x4{0, 0, 0, 0};

    // Each wave walks k-steps wave, wave + KW, ... of the range on its own:
    // its LDS area is private, so only wave-level ordering is needed (LDS
    // operations of one wave complete in order).
    uint32_t wc[16], wn[16];
    int w = w_begin + wave;
    if (w < w_end) {
        load_w(w, wc);
        stage(load_bits(w));
    }
    for (; w < w_end; w += KW) {
        const bool more = w + KW < w_end;
        uint64_t nbits = 0;
        if (more) {
            load_w(w + KW, wn);
            nbits = load_bits(w + KW);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        mf_i32x4 a[4];
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
            a[ms] = *reinterpret_cast<const mf_i32x4*>(&xw[(ms * 16 + c) * kXPitch + q * 16]);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        __builtin_amdgcn_wave_barrier();
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
        if (more)
            stage(nbits);  // the A-operands of this step are already in registers
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                acc[ms][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ms], f[t], acc[ms][t], 0, 0, 0);
        if (more) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
                wc[i] = wn[i];
        }
    }

    __syncthreads();  // red is zeroed everywhere
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                atomicAdd(&red[(16 * ms + 4 * q + j) * kMfmaCols + 4 * c + t], acc[ms][t][j]);
    __syncthreads();

    auto write_tile = [&](auto value_at) {
        for (int e = threadIdx.x; e < TILE; e += BLOCK) {
            const int b = m0 + e / kMfmaCols;
            const int64_t n = n0 + e % kMfmaCols;
            if (b < B) {
                const int32_t sum = value_at(e);
                if constexpr (ACC) {
                    acc_out[(int64_t)b * N + n] = sum;
                } else {
                    const float as_float = (float)sum;  // exact for |sum| < 2^24, RNE beyond
                    out[(int64_t)b * N + n] = as_float * scale[n];
                }
            }
        }
    };
    if (n_splits == 1) {
        write_tile([&](int e) { return red[e]; });
        return;
    }

    // K split across workgroups (only with a single row tile, B <= 64):
    // each split stores the B valid rows of its partial tile with plain
    // stores; the last split to arrive (completion counter) adds them.
    const int valid = B * kMfmaCols;  // rows of this tile that exist
    int32_t* my_part = parts + ((int64_t)tile_id * n_splits + split) * valid;
    for (int e = threadIdx.x; e < valid; e += BLOCK)
        __hip_atomic_store(my_part + e, red[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    wait_writes_done();  // the partial tile is stored before it is counted
    __syncthreads();
    uint32_t* counter = counters + tile_id;
    if (threadIdx.x == 0)
        is_last = atomicAdd(counter, 1u) == (uint32_t)(n_splits - 1);
    __syncthreads();
    if (!is_last)
        return;
    int32_t* tile_parts = parts + (int64_t)tile_id * n_splits * valid;
    write_tile([&](int e) {
        int32_t sum = 0;
        for (int sidx = 0; sidx < n_splits; ++sidx)
            sum += __hip_atomic_load(tile_parts + (int64_t)sidx * valid + e, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
        return sum;
    });
    if (threadIdx.x == 0)
        atomicExch(counter, 0u);
}

// Launch over B rows.  A workgroup owns a 64 x 64 tile; when the tiles alone
// cannot fill the chip (B <= 64: one row tile), K is split across workgroups
// so that about 256 run, up to kMfmaMaxSplits (words_per_split_req > 0 fixes
// the split).  Splitting needs B <= 64, N/64 zeroed counters and a
// partial-tile area of n_splits * B * N INT32.
constexpr int kMfmaMaxSplits = 8;
constexpr int kMfmaSplitRows = 64;  // splits are used only up to this many rows

inline int mfma_splits(int K, int N, int B, int words_per_split_req, int* wps_out)
{
    const int wpr = (K + 63) / 64;
    const int tiles = ((B + kMfmaRows - 1) / kMfmaRows) * (N / kMfmaCols);
    int wps;
    (void)tiles;
    if (words_per_split_req > 0) {
        wps = words_per_split_req;
    } else if (B <= kMfmaSplitRows) {
        // measured: about three 64-wide k-steps per wave of an 8-wave
        // workgroup is best for up to 32 rows, six for up to 64 rows
        wps = B <= 32 ? 24 : 48;
        const int min_wps = (wpr + kMfmaMaxSplits - 1) / kMfmaMaxSplits;
        wps = wps < min_wps ? min_wps : wps;
    } else {
        wps = wpr;  // enough row tiles to fill the chip
    }
    wps = wps > wpr ? wpr : (wps < 1 ? 1 : wps);
    *wps_out = wps;
    return (wpr + wps - 1) / wps;
}

template <int KW>
hipError_t launch_mfma_t(const int8_t* W, const float* scale, int K, int N, const uint64_t* mask, int B, int wps,
                         int n_splits, int32_t* parts, uint32_t* counters, float* out, int32_t* acc, bool want_acc,
                         hipStream_t st)
{
    const int wpr = (K + 63) / 64;
    const int n_coltiles = N / kMfmaCols;
    const int n_rowtiles = (B + kMfmaRows - 1) / kMfmaRows;
    const int64_t units = (int64_t)n_coltiles * n_rowtiles * n_splits;
    if (units > 0x7fffffff)
        return hipErrorInvalidValue;
    if (want_acc)
        hipLaunchKernelGGL((k_mfma<KW, true>), dim3((unsigned)units), dim3(64 * KW), 0, st, W, scale, K, N, mask,
                           wpr, B, wps, n_splits, n_coltiles, parts, counters, out, acc);
    else
        hipLaunchKernelGGL((k_mfma<KW, false>), dim3((unsigned)units), dim3(64 * KW), 0, st, W, scale, K, N, mask,
                           wpr, B, wps, n_splits, n_coltiles, parts, counters, out, acc);
    return hipGetLastError();
}

// waves_req: 0 = automatic (8 waves per workgroup share a tile's K range,
// measured best or equal at every batch size tried).
inline hipError_t launch_mfma(const int8_t* W, const float* scale, int K, int N, const uint64_t* mask, int B,
                              int wps, int n_splits, int waves_req, int32_t* parts, uint32_t* counters, float* out,
                              int32_t* acc, bool want_acc, hipStream_t st)
{
    const int waves = waves_req == 0 ? 8 : waves_req;
    switch (waves) {
    case 4: return launch_mfma_t<4>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc, want_acc, st);
    case 8: return launch_mfma_t<8>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc, want_acc, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace spk
