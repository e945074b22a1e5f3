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
constexpr int kXRow = 64;        // LDS bytes per expanded spike row (quarters swizzled)
constexpr int kMfmaDefaultDepth = 2;  // k-steps of weights in flight per wave

typedef int32_t mf_i32x4 __attribute__((ext_vector_type(4)));

constexpr int kBufferWordFormat = 0x00020000;  // buffer resource word 3: 32-bit data format (gfx9)

// The weight matrix must be addressable by 32-bit byte offsets (one buffer
// resource): K * N < 2^31.
inline bool mfma_supported(int K, int N, const void* W)
{
    return N % kMfmaNAlign == 0 && reinterpret_cast<uintptr_t>(W) % 4 == 0 && (int64_t)K * N < (1ll << 31);
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

template <int KW, int D, int NS, bool ACC>
__global__ __launch_bounds__(64 * KW) void k_mfma(const int8_t* __restrict__ W, const float* __restrict__ scale,
                                                  int K, int N, const uint64_t* __restrict__ mask, int wpr, int B,
                                                  int words_per_split, int n_splits, int n_coltiles,
                                                  int32_t* __restrict__ parts, uint32_t* counters, float* out,
                                                  int32_t* acc_out)
{
    constexpr int BLOCK = 64 * KW;
    constexpr int TILE = kMfmaRows * kMfmaCols;
    __shared__ __align__(16) uint8_t xs[KW][kMfmaRows * kXRow];  // one area per wave
    __shared__ int32_t red[TILE];                                  // the tile's INT32 sums
    __shared__ int32_t is_last;

    // wave index as a scalar, so that everything derived from it (k-steps,
    // buffer offsets) is known to be uniform across the wave
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
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
    __syncthreads();

    uint8_t* xw = xs[wave];
    const int xb = m0 + l;  // the row this lane stages
    // W: 4 channels (n0 + 4c ..) of k-rows kb + 16q + i, i < 16.  For a full
    // step the row base of each i is the same in every lane (a scalar
    // register) and the lane adds a 32-bit offset, so the addresses cost no
    // vector ALU; in the last, partial step rows past K are clamped to a
    // valid row (their spikes are zero).
    // Buffer loads: the weight matrix is one buffer resource (scalar
    // registers), the lane adds a fixed 32-bit offset and each of the 16
    // rows a scalar offset, so the addresses cost no vector ALU.  Offsets at
    // or past K*N (rows beyond K in the last step) read 0 instead of memory.
    const __amdgpu_buffer_rsrc_t wrsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(W), 0, K * N, kBufferWordFormat);
    const int lane_off = 16 * q * N + 4 * c;
    auto load_w = [&](int w, uint32_t (&d)[16]) {
        const int row0 = w * kMfmaK * N + n0;
#pragma unroll
        for (int i = 0; i < 16; ++i)
            d[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(wrsrc, lane_off, row0 + i * N, 0);
    };
    // The raw word is kept in flight; bits at or above K are cleared only
    // when it is staged, so that issuing the load never waits for it.
    auto load_bits = [&](int w) -> uint64_t { return xb < B ? mask[(int64_t)xb * wpr + w] : 0ull; };
    // this lane's row of the wave's LDS area <- the 64 spikes of step w as
    // 0/1 bytes.  Rows are 64 bytes; the four 16-byte quarters of row r sit
    // at quarter slot q ^ ((r >> 1) & 3), which makes both the row writes
    // here and the operand reads below free of LDS bank conflicts (any 8
    // consecutive lanes touch all 32 banks once).
    auto stage = [&](uint64_t word, int w) {
        const int valid = K - 64 * w;
        if (valid < 64)
            word &= valid <= 0 ? 0ull : ((1ull << valid) - 1ull);
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const uint32_t bits = (uint32_t)(word >> (16 * qq));
            uint4 v;
            v.x = expand_nibble(bits);
            v.y = expand_nibble(bits >> 4);
            v.z = expand_nibble(bits >> 8);
            v.w = expand_nibble(bits >> 12);
            *reinterpret_cast<uint4*>(&xw[l * kXRow + ((qq ^ ((l >> 1) & 3)) * 16)]) = v;
        }
    };

    mf_i32x4 acc[4][4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int t = 0; t < 4; ++t)
            acc[ms][t] = mf_i32x4{0, 0, 0, 0};

    // Each wave walks k-steps wave, wave + KW, ... of the range on its own,
    // with the weights and spike words of the next D steps in flight (a ring
    // of D register slots; the loop is unrolled by D so slot indices stay
    // static).  The wave's LDS area is private, so only wave-level ordering
    // is needed (LDS operations of one wave complete in order).
    const int n_steps = w_begin + wave < w_end ? (w_end - w_begin - wave + KW - 1) / KW : 0;
    // Loads are issued unconditionally, for a step index clamped to the
    // wave's last step (extra loads re-read cached data): a conditional
    // refill would turn the ring slots into phis that the compiler fills
    // with copies, and every copy waits for its load.
    const int last_w = w_begin + wave + (n_steps - 1) * KW;
    auto step_w = [&](int i) { return min(w_begin + wave + i * KW, last_w); };
    uint32_t wbuf[D][16];
    uint64_t bits[D];
    // one k-step: consume ring slot d (step i), refill it with step i + D
    auto step = [&](int d, int i, bool live) {
        stage(live ? bits[d] : 0ull, step_w(i));
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        mf_i32x4 a[4];
#pragma unroll
        for (int ms = 0; ms < 4; ++ms) {
            const int r = ms * 16 + c;
            a[ms] = *reinterpret_cast<const mf_i32x4*>(&xw[r * kXRow + ((q ^ ((r >> 1) & 3)) * 16)]);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        mf_i32x4 f[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            uint32_t e0, e1, e2, e3;
            transpose4x4(wbuf[d][4 * m], wbuf[d][4 * m + 1], wbuf[d][4 * m + 2], wbuf[d][4 * m + 3], e0, e1, e2, e3);
            f[0][m] = (int32_t)e0;
            f[1][m] = (int32_t)e1;
            f[2][m] = (int32_t)e2;
            f[3][m] = (int32_t)e3;
        }
        // Keep the refill below the transposes that read the old slot: if the
        // scheduler hoists it, old and new values live in different
        // registers and the ring turns into copies that wait for the loads.
        __builtin_amdgcn_sched_barrier(0);
        load_w(step_w(i + D), wbuf[d]);
        bits[d] = load_bits(step_w(i + D));
        if (live) {
#pragma unroll
            for (int ms = 0; ms < 4; ++ms)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    acc[ms][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ms], f[t], acc[ms][t], 0, 0, 0);
        }
    };
    if (n_steps > 0) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            load_w(step_w(d), wbuf[d]);
            bits[d] = load_bits(step_w(d));
        }
        if (NS > 0 && n_steps == NS) {
            // The common step counts are unrolled completely: with no loop
            // back-edge there are no phis for the compiler to fill with
            // copies of the ring that wait for their loads.
#pragma unroll
            for (int i = 0; i < NS; ++i)
                step(i % D, i, true);
        } else {
            const int n_full = n_steps / D * D;
            int i0 = 0;
            for (; i0 < n_full; i0 += D) {
#pragma unroll
                for (int d = 0; d < D; ++d)
                    step(d, i0 + d, true);
            }
#pragma unroll
            for (int d = 0; d < D; ++d)
                if (i0 + d < n_steps)
                    step(d, i0 + d, true);
        }
    }

    __syncthreads();  // every wave is done with its steps
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

template <int KW, int D, int NS>
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
        hipLaunchKernelGGL((k_mfma<KW, D, NS, true>), dim3((unsigned)units), dim3(64 * KW), 0, st, W, scale, K, N,
                           mask, wpr, B, wps, n_splits, n_coltiles, parts, counters, out, acc);
    else
        hipLaunchKernelGGL((k_mfma<KW, D, NS, false>), dim3((unsigned)units), dim3(64 * KW), 0, st, W, scale, K, N,
                           mask, wpr, B, wps, n_splits, n_coltiles, parts, counters, out, acc);
    return hipGetLastError();
}

// waves_req: 0 = automatic (8 waves per workgroup share a tile's K range,
// measured best or equal at every batch size tried).  depth_req: k-steps in
// flight per wave, 0 = automatic.  The step counts per wave that the
// automatic splits produce (3, 6, 12 for 8 waves) get fully unrolled kernels.
inline hipError_t launch_mfma(const int8_t* W, const float* scale, int K, int N, const uint64_t* mask, int B,
                              int wps, int n_splits, int waves_req, int depth_req, int32_t* parts,
                              uint32_t* counters, float* out, int32_t* acc, bool want_acc, hipStream_t st)
{
    const int waves = waves_req == 0 ? 8 : waves_req;
    const int depth = depth_req == 0 ? kMfmaDefaultDepth : depth_req;
    // steps per wave when every split spans wps words (the last split may be shorter)
    const int wpr = (K + 63) / 64;
    const bool uniform = wpr % wps == 0;
    const int ns = uniform && wps % waves == 0 ? wps / waves : 0;
#define SPK_MFMA_CASE(KW, D)                                                                                       \
    if (waves == KW && depth == D) {                                                                               \
        if (ns == 3)                                                                                               \
            return launch_mfma_t<KW, D, 3>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,      \
                                           want_acc, st);                                                          \
        if (ns == 6)                                                                                               \
            return launch_mfma_t<KW, D, 6>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,      \
                                           want_acc, st);                                                          \
        if (ns == 12)                                                                                              \
            return launch_mfma_t<KW, D, 12>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,     \
                                            want_acc, st);                                                         \
        return launch_mfma_t<KW, D, 0>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,          \
                                       want_acc, st);                                                              \
    }
    SPK_MFMA_CASE(4, 1)
    SPK_MFMA_CASE(4, 2)
    SPK_MFMA_CASE(8, 1)
    SPK_MFMA_CASE(8, 2)
#undef SPK_MFMA_CASE
    // four steps in flight: generic loop only (unrolled, it runs out of registers)
    if (depth == 4 && waves == 4)
        return launch_mfma_t<4, 4, 0>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc, want_acc,
                                      st);
    if (depth == 4 && waves == 8)
        return launch_mfma_t<8, 4, 0>(W, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc, want_acc,
                                      st);
    return hipErrorInvalidValue;
}

}  // namespace spk
