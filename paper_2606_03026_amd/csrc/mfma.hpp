// Dense i8 matrix-core contraction over the 0/1 spike matrix, for batches of
// spike rows (gfx950 v_mfma_i32_16x16x64_i8).
//
// For B spike rows the projection of Eq. (sparse) (paper Sec. 2.3) is the
// integer product acc[b][n] = sum_k x[b][k] * Q[n][k] with x in {0,1}; the
// matrix cores compute it densely (every column is read once per row tile
// instead of once per active (row, column) pair) and it stays exact: every
// product is 0 or a weight, and INT32 sums are exact.  The FP32 epilogue is
// the same single conversion and multiply as the gather path, so both paths
// give identical bits.
//
// Operand layout.  The matrix core wants, in every lane, 16 consecutive k of
// one output channel; the column-major W of the gather path has consecutive
// channels in consecutive bytes instead.  A handle therefore keeps a packed
// copy of W, made once when it is created, in exactly the operand order:
//
//   [N/64 column tiles][ceil(K/64) k-steps][4 channel sets][64 lanes][16 B]
//
// where lane l = 16q + c of channel set t of column tile ct, k-step s holds
// W[64s + 16q + j][64ct + 16t + c] in byte j (zero for k >= K).  One k-step
// of one column tile is 4 KB of contiguous memory, every lane fetches its
// B-operand with one 16-byte load, and a column tile's whole K range is one
// contiguous run.  Spike bits past K meet zero weights there, so the mask
// needs no trimming.  The A-operand of row r, k = 16q .. 16q + 15 is built
// in registers from bits 16q .. 16q + 15 of the row's mask word (one byte of
// 0 or 1 per bit).  The mask words are staged in LDS first, a chunk of the
// workgroup's K range for all its 64 rows with coalesced loads: loaded from
// global memory per k-step, each wave's words would come from 16 rows at
// once, and such scattered loads measured twice as slow as the whole rest
// of the kernel.  Result layout of the 16x16 i32 accumulator (checked on
// the device): lane l, register j holds row 4*(l/16) + j, column l%16.
//
// Work split.  A workgroup owns one 64-row x 64-channel tile; its KW waves
// take interleaved k-steps of the workgroup's K range, each with the next D
// steps' loads in flight, and their partial tiles are added through LDS in
// a two-level tree.  When the tiles alone cannot fill the chip (B <= 64), K
// is also split across workgroups: each stores its partial tile, and the
// last to arrive (one counter atomic per workgroup) adds them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "gather.hpp"  // wait_writes_done, u32x4

namespace spk {

constexpr int kMfmaNAlign = 64;  // N must be a multiple of this
constexpr int kMfmaRows = 64;    // spike rows per tile (4 subtiles of 16)
constexpr int kMfmaCols = 64;    // channels per tile (4 MFMA channel sets of 16)
constexpr int kMfmaK = 64;       // k per step: one mask word
constexpr int kMfmaStepBytes = kMfmaK * kMfmaCols;  // one k-step of one column tile in the packed copy
constexpr int kMfmaGroups = 16 * 64;                // 4-entry groups of a tile: (row set, channel set, lane)
constexpr int kMfmaDefaultDepth = 2;                // k-steps of loads in flight per wave
constexpr int kMfmaStageWords = 96;                 // mask words per row staged in LDS at a time
constexpr int kMfmaStagePitch = kMfmaStageWords + 1;  // padded row pitch (words): conflict-free reads

typedef int32_t mf_i32x4 __attribute__((ext_vector_type(4)));

constexpr int kBufferWordFormat = 0x00020000;  // buffer resource word 3: 32-bit data format (gfx9)
// Cache policy of buffer loads and stores that must be coherent across the
// XCDs' L2 caches: sc1, the policy of device-scope atomic loads and stores.
constexpr int kCoherent = 16;

// Bytes of the packed copy of a K x N matrix.
inline int64_t mfma_packed_bytes(int64_t K, int64_t N) { return (K + kMfmaK - 1) / kMfmaK * kMfmaK * N; }

// The packed copy must be addressable by 31-bit byte offsets (one buffer
// resource) and N must split into whole column tiles.
inline bool mfma_supported(int64_t K, int64_t N)
{
    return N % kMfmaNAlign == 0 && mfma_packed_bytes(K, N) < (1ll << 31);
}

// One thread per 16-byte lane chunk of the packed copy.
constexpr int kPackBlock = 256;
__global__ __launch_bounds__(kPackBlock) void k_mfma_pack(const int8_t* __restrict__ W, int K, int N, int wpr,
                                                          int8_t* __restrict__ P, int64_t n_chunks)
{
    const int64_t id = (int64_t)blockIdx.x * kPackBlock + threadIdx.x;
    if (id >= n_chunks)
        return;
    const int l = (int)(id % 64);
    const int t = (int)((id / 64) % 4);
    const int64_t ts = id / 256;  // column tile * wpr + k-step
    const int64_t s = ts % wpr;
    const int64_t ct = ts / wpr;
    const int64_t n = ct * kMfmaCols + 16 * t + l % 16;
    const int64_t k0 = kMfmaK * s + 16 * (l / 16);
    uint32_t v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t w = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int64_t k = k0 + 4 * i + b;
            const uint32_t byte = k < K ? (uint32_t)(uint8_t)W[k * N + n] : 0u;
            w |= byte << (8 * b);
        }
        v[i] = w;
    }
    *reinterpret_cast<u32x4*>(P + id * 16) = u32x4{v[0], v[1], v[2], v[3]};
}

// Four spike bits -> four bytes holding 0 or 1 (bit i -> byte i).
__device__ inline uint32_t expand_nibble(uint32_t bits) { return ((bits & 0xFu) * 0x00204081u) & 0x01010101u; }

template <int KW, int D, int NS, bool ACC>
__global__ __launch_bounds__(64 * KW) void k_mfma(const int8_t* __restrict__ P, const float* __restrict__ scale,
                                                  int N, const uint64_t* __restrict__ mask, int wpr, int B,
                                                  int words_per_split, int n_splits, int n_coltiles,
                                                  int32_t* __restrict__ parts, uint32_t* counters, float* out,
                                                  int32_t* acc_out)
{
    static_assert(KW == 4 || KW == 8, "four or eight waves per workgroup");
    constexpr int BLOCK = 64 * KW;
    constexpr int PER = kMfmaGroups / BLOCK;  // result groups per thread in the final sum
    // LDS: the staged mask words while the k-steps run, then the four
    // partial tiles of the reduction tree
    constexpr int kRedBytes = 4 * kMfmaGroups * (int)sizeof(mf_i32x4);
    static_assert(kMfmaRows * kMfmaStagePitch * (int)sizeof(uint64_t) <= kRedBytes, "stage fits the tree area");
    __shared__ __align__(16) uint8_t lds[kRedBytes];
    auto red = reinterpret_cast<mf_i32x4(*)[kMfmaGroups]>(lds);
    uint64_t* xs = reinterpret_cast<uint64_t*>(lds);
    __shared__ int32_t is_last;

    // wave index as a scalar, so that everything derived from it (k-steps,
    // buffer offsets) is known to be uniform across the wave
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int l = threadIdx.x % 64;
    const int q = l / 16;  // k-group of the operands, row group of the result
    const int c = l % 16;  // row of A, channel of B and of the result
    const int split = blockIdx.x % n_splits;
    const int tile_id = blockIdx.x / n_splits;
    const int ct = tile_id % n_coltiles;
    const int rt = tile_id / n_coltiles;
    const int m0 = rt * kMfmaRows;
    const int n0 = ct * kMfmaCols;
    const int w_begin = split * words_per_split;
    const int w_end = min(wpr, w_begin + words_per_split);

    // The weight copy is a buffer resource: the lane's offset is a fixed
    // vector register, the k-step a scalar, so addressing costs no vector ALU.
    const __amdgpu_buffer_rsrc_t prsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t*>(P), 0, n_coltiles * wpr * kMfmaStepBytes, kBufferWordFormat);
    const int tile_step0 = ct * wpr;
    auto load_w = [&](int s, u32x4 (&wv)[4]) {
        const int base = (tile_step0 + s) * kMfmaStepBytes;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            wv[t] = __builtin_amdgcn_raw_buffer_load_b128(prsrc, 16 * l + 1024 * t, base, 0);
    };
    // mask words [w0, w0 + nw) of the tile's 64 rows -> xs.  Wave v takes
    // rows v, v + KW, ..., its lanes consecutive words; every load is issued
    // before the first store.  The mask is a buffer resource, so rows at or
    // past B read as 0.
    static_assert(kMfmaStageWords <= 128, "two words per lane and row");
    const __amdgpu_buffer_rsrc_t mrsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint64_t*>(mask), 0, B * wpr * (int)sizeof(uint64_t), kBufferWordFormat);
    auto stage = [&](int w0, int nw) {
        constexpr int RPW = kMfmaRows / KW;  // rows per wave
        u32x2 v[RPW][2];
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int w = min(l + 64 * h, nw - 1);
                v[rr][h] = __builtin_amdgcn_raw_buffer_load_b64(
                    mrsrc, ((m0 + wave + rr * KW) * wpr + w) * (int)sizeof(uint64_t), w0 * (int)sizeof(uint64_t), 0);
            }
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                if (l + 64 * h < nw)
                    xs[(wave + rr * KW) * kMfmaStagePitch + l + 64 * h] = __builtin_bit_cast(uint64_t, v[rr][h]);
    };
    // Spikes 16q .. 16q + 15 of row 16 ms + c for staged word w: one 16-bit
    // LDS read per row set (the 16 rows of a read sit in distinct banks
    // thanks to the odd row pitch), expanded to the A-operand bytes.
    const uint16_t* xs16 = reinterpret_cast<const uint16_t*>(xs);
    auto read_bits = [&](int w, uint32_t (&b16)[4]) {
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
            b16[ms] = xs16[((16 * ms + c) * kMfmaStagePitch + w) * 4 + q];
    };
    auto operand_a = [&](uint32_t b16) {
        return mf_i32x4{(int32_t)expand_nibble(b16), (int32_t)expand_nibble(b16 >> 4),
                        (int32_t)expand_nibble(b16 >> 8), (int32_t)expand_nibble(b16 >> 12)};
    };

    mf_i32x4 acc[4][4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int t = 0; t < 4; ++t)
            acc[ms][t] = mf_i32x4{0, 0, 0, 0};

    // Per staged chunk, each wave walks k-steps wave, wave + KW, ... of the
    // chunk with the weight loads of the next D steps in flight (a ring of D
    // register slots; the loop is unrolled by D so slot indices stay
    // static).  Loads are issued unconditionally, for a step index clamped
    // to the wave's last step (extra loads re-read cached data): a
    // conditional refill would turn the ring slots into phis that the
    // compiler fills with copies, and every copy waits for its load.
    int cw0 = w_begin, n_steps = 0, last_w = 0;
    auto step_w = [&](int i) { return min(cw0 + wave + i * KW, last_w); };
    u32x4 wbuf[D][4];
    uint32_t bits[4];  // spike bits of the next step, read one step ahead
    // One k-step: consume ring slot d (step i) and refill it with step i + D.
    // Refilled before the products (early), a load is covered by D steps of
    // work; the old and new contents of the slot are then live together,
    // which costs nothing where the steps are unrolled completely but turns
    // into register copies (each waiting for its load) at a loop back-edge.
    // In the loop the refill therefore follows the products and reuses the
    // slot's registers (D - 1 steps of cover).
    auto step = [&](int d, int i, auto early) {
        __builtin_amdgcn_sched_barrier(0);
        mf_i32x4 a[4];
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
            a[ms] = operand_a(bits[ms]);
        mf_i32x4 f[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
            f[t] = __builtin_bit_cast(mf_i32x4, wbuf[d][t]);
        __builtin_amdgcn_sched_barrier(0);
        // the next step's spike bits (its LDS latency hides behind the products)
        read_bits(min(wave + (i + 1) * KW, last_w - cw0), bits);
        if constexpr (decltype(early)::value)
            load_w(step_w(i + D), wbuf[d]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                acc[ms][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ms], f[t], acc[ms][t], 0, 0, 0);
        if constexpr (!decltype(early)::value) {
            __builtin_amdgcn_sched_barrier(0);
            load_w(step_w(i + D), wbuf[d]);
        }
    };
    using Early = std::true_type;
    using Late = std::false_type;
    for (; cw0 < w_end; cw0 += kMfmaStageWords) {
        const int cw = min(kMfmaStageWords, w_end - cw0);
        n_steps = wave < cw ? (cw - wave + KW - 1) / KW : 0;
        last_w = cw0 + wave + (n_steps - 1) * KW;
        if (n_steps > 0) {
#pragma unroll
            for (int d = 0; d < D; ++d)
                load_w(step_w(d), wbuf[d]);  // in flight while the chunk is staged
        }
        stage(cw0, cw);
        __syncthreads();
        if (n_steps > 0)
            read_bits(wave, bits);
        if constexpr (NS > 0) {
            // The common step counts are unrolled completely.  Such a kernel
            // is launched only where every wave has exactly NS k-steps in a
            // single chunk (and holds no generic loop: its registers would
            // be the union of both paths').
#pragma unroll
            for (int i = 0; i < NS; ++i)
                step(i % D, i, Early{});
        } else if (n_steps > 0) {
            const int n_full = n_steps / D * D;
            int i0 = 0;
            for (; i0 < n_full; i0 += D) {
#pragma unroll
                for (int d = 0; d < D; ++d)
                    step(d, i0 + d, Late{});
            }
#pragma unroll
            for (int d = 0; d < D; ++d)
                if (i0 + d < n_steps)
                    step(d, i0 + d, Late{});
        }
        __syncthreads();  // the chunk's staged words are read before they are replaced
    }

    // Reduction tree over the waves' partial tiles, in register order
    // (group (ms * 4 + t) * 64 + lane holds the lane's four registers of
    // accumulator (ms, t)): waves 4..7 hand theirs to waves 0..3, then
    // waves 0..3 store and every thread adds the four tiles for its groups.
    auto put = [&](int slot) {
#pragma unroll
        for (int ms = 0; ms < 4; ++ms)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                red[slot][(ms * 4 + t) * 64 + l] = acc[ms][t];
    };
    if constexpr (KW == 8) {
        if (wave >= 4)
            put(wave - 4);
        __syncthreads();
        if (wave < 4) {
#pragma unroll
            for (int ms = 0; ms < 4; ++ms)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    acc[ms][t] += red[wave][(ms * 4 + t) * 64 + l];
        }
        __syncthreads();
    }
    if (wave < 4)
        put(wave);
    __syncthreads();
    mf_i32x4 sum[PER];
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int g = threadIdx.x + r * BLOCK;
        sum[r] = red[0][g] + red[1][g] + red[2][g] + red[3][g];
    }

    // group g -> rows m0 + 16 ms + 4 (g%64 / 16) + j, channel n0 + 16 t + g%16
    auto write_groups = [&](const mf_i32x4 (&v)[PER]) {
#pragma unroll
        for (int r = 0; r < PER; ++r) {
            const int g = threadIdx.x + r * BLOCK;
            const int mt = g / 64, lg = g % 64;
            const int row0 = m0 + 16 * (mt / 4) + 4 * (lg / 16);
            const int64_t n = n0 + 16 * (mt % 4) + lg % 16;
            float sc = 0.0f;
            if constexpr (!ACC)
                sc = scale[n];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int b = row0 + j;
                if (b < B) {
                    if constexpr (ACC) {
                        acc_out[(int64_t)b * N + n] = v[r][j];
                    } else {
                        const float as_float = (float)v[r][j];  // exact for |sum| < 2^24, RNE beyond
                        out[(int64_t)b * N + n] = as_float * sc;
                    }
                }
            }
        }
    };
    if (n_splits == 1) {
        write_groups(sum);
        return;
    }

    // K split across workgroups (one row tile, B <= 64): every split stores
    // its partial tile (device-coherent stores); the last split to arrive
    // (completion counter) loads the others, all loads in flight at once.
    const __amdgpu_buffer_rsrc_t parts_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        parts, 0, n_coltiles * n_splits * kMfmaGroups * (int)sizeof(mf_i32x4), kBufferWordFormat);
    const int tile_part0 = tile_id * n_splits;
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int g = threadIdx.x + r * BLOCK;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, sum[r]), parts_rsrc,
                                               (int)sizeof(mf_i32x4) * g,
                                               (tile_part0 + split) * kMfmaGroups * (int)sizeof(mf_i32x4),
                                               kCoherent);
    }
    wait_writes_done();  // the partial tile is stored before it is counted
    __syncthreads();
    uint32_t* counter = counters + tile_id;
    if (threadIdx.x == 0)
        is_last = atomicAdd(counter, 1u) == (uint32_t)(n_splits - 1);
    __syncthreads();
    if (!is_last)
        return;
    constexpr int kMaxParts = 8;
    mf_i32x4 other[kMaxParts][PER];
#pragma unroll
    for (int sidx = 0; sidx < kMaxParts; ++sidx) {
        const int src = min(sidx, n_splits - 1);
#pragma unroll
        for (int r = 0; r < PER; ++r) {
            const int g = threadIdx.x + r * BLOCK;
            other[sidx][r] = __builtin_bit_cast(
                mf_i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                              parts_rsrc, (int)sizeof(mf_i32x4) * g,
                              (tile_part0 + src) * kMfmaGroups * (int)sizeof(mf_i32x4), kCoherent));
        }
    }
#pragma unroll
    for (int sidx = 0; sidx < kMaxParts; ++sidx) {
        const bool use = sidx < n_splits && sidx != split;
#pragma unroll
        for (int r = 0; r < PER; ++r)
            sum[r] += use ? other[sidx][r] : mf_i32x4{0, 0, 0, 0};
    }
    write_groups(sum);
    if (threadIdx.x == 0)
        atomicExch(counter, 0u);
}

// Launch over B rows.  A workgroup owns a 64 x 64 tile; when the tiles alone
// cannot fill the chip (B <= 64: one row tile), K is split across workgroups
// up to kMfmaMaxSplits (words_per_split_req > 0 fixes the split).  Splitting
// needs B <= 64, N/64 zeroed counters and a partial-tile area of
// n_splits * 64 * N INT32.
constexpr int kMfmaMaxSplits = 8;
constexpr int kMfmaSplitRows = 64;  // splits are used only up to this many rows

inline int mfma_splits(int K, int N, int B, int words_per_split_req, int* wps_out)
{
    const int wpr = (K + 63) / 64;
    int wps;
    (void)N;
    if (words_per_split_req > 0) {
        wps = words_per_split_req;
    } else if (B <= kMfmaSplitRows) {
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
hipError_t launch_mfma_t(const int8_t* P, const float* scale, int K, int N, const uint64_t* mask, int B, int wps,
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
        hipLaunchKernelGGL((k_mfma<KW, D, NS, true>), dim3((unsigned)units), dim3(64 * KW), 0, st, P, scale, N,
                           mask, wpr, B, wps, n_splits, n_coltiles, parts, counters, out, acc);
    else
        hipLaunchKernelGGL((k_mfma<KW, D, NS, false>), dim3((unsigned)units), dim3(64 * KW), 0, st, P, scale, N,
                           mask, wpr, B, wps, n_splits, n_coltiles, parts, counters, out, acc);
    return hipGetLastError();
}

// waves_req: 0 = automatic (8 waves per workgroup).  depth_req: k-steps in
// flight per wave, 0 = automatic.  The step counts per wave that the
// automatic splits produce (3, 6, 12 for 8 waves) get fully unrolled kernels.
inline hipError_t launch_mfma(const int8_t* P, const float* scale, int K, int N, const uint64_t* mask, int B,
                              int wps, int n_splits, int waves_req, int depth_req, int32_t* parts,
                              uint32_t* counters, float* out, int32_t* acc, bool want_acc, hipStream_t st)
{
    const int waves = waves_req == 0 ? 8 : waves_req;
    const int depth = depth_req == 0 ? kMfmaDefaultDepth : depth_req;
    // k-steps per wave when every workgroup's range is wps words, staged as
    // one chunk, shared evenly by the waves; otherwise the generic loop
    const int wpr = (K + 63) / 64;
    const bool uniform = wpr % wps == 0 && wps <= kMfmaStageWords;
    const int ns = uniform && wps % waves == 0 ? wps / waves : 0;
#define SPK_MFMA_CASE(KW, D)                                                                                       \
    if (waves == KW && depth == D) {                                                                               \
        if (ns == 3)                                                                                               \
            return launch_mfma_t<KW, D, 3>(P, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,      \
                                           want_acc, st);                                                          \
        if (ns == 6)                                                                                               \
            return launch_mfma_t<KW, D, 6>(P, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,      \
                                           want_acc, st);                                                          \
        if (ns == 12)                                                                                              \
            return launch_mfma_t<KW, D, 12>(P, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,     \
                                            want_acc, st);                                                         \
        return launch_mfma_t<KW, D, 0>(P, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc,          \
                                       want_acc, st);                                                              \
    }
    SPK_MFMA_CASE(4, 1)
    SPK_MFMA_CASE(4, 2)
    SPK_MFMA_CASE(8, 1)
    SPK_MFMA_CASE(8, 2)
#undef SPK_MFMA_CASE
    // four steps in flight: generic loop only
    if (depth == 4 && waves == 4)
        return launch_mfma_t<4, 4, 0>(P, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc, want_acc,
                                      st);
    if (depth == 4 && waves == 8)
        return launch_mfma_t<8, 4, 0>(P, scale, K, N, mask, B, wps, n_splits, parts, counters, out, acc, want_acc,
                                      st);
    return hipErrorInvalidValue;
}

}  // namespace spk
