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
// copy of W in exactly the operand order, one 16-channel set after another:
//
//   [N/16 channel sets][ceil(K/64) k-steps][64 lanes][16 B]
//
// where lane l = 16q + c of channel set t, k-step s holds
// W[64s + 16q + j][16t + c] in byte j (zero for k >= K).  One k-step of one
// channel set is 1 KB of contiguous memory, every lane fetches its B-operand
// with one 16-byte load, and a channel set's whole K range is one contiguous
// run.  Spike bits past K meet zero weights there, so the mask needs no
// trimming.  The A-operand of row r, k = 16q .. 16q + 15 is built in
// registers from bits 16q .. 16q + 15 of the row's mask word (one byte of 0
// or 1 per bit).  The workgroup first stages the mask words of its rows in
// LDS with coalesced loads (row pitch odd in words, so that the 16 rows of
// one operand read sit in distinct banks); for batches of at most 4 rows each
// lane instead loads the dword holding its 16 bits with each k-step's
// weights (DIRECT plans).  Result layout of the 16x16 i32
// accumulator (checked on the device): lane l, register j holds row
// 4*(l/16) + j, column l%16.
//
// Work split.  A workgroup owns a tile of RT row subtiles (16 rows each) by
// CS channel sets (16 channels each) over the whole K range; its KW waves
// take interleaved k-steps and add their partial tiles with LDS atomics
// (integer, so the order does not matter).  Nothing crosses workgroups, so
// a launch needs no workspace and no cross-workgroup hand-off.  Small
// batches are spread over the chip by narrow tiles (one 16-row subtile by
// one channel set); the row tiles that share a channel set are placed on the
// same XCD so that its weights come from HBM once and from that XCD's L2
// after.  Large batches use tall tiles so that each weight byte fetched into
// a compute unit feeds RT * 16 rows.
//
// Weight loads: with D >= the wave's k-step count (PRELOAD) every load of
// the wave is issued before the spike words are staged, so a small tile
// costs one memory round trip; otherwise the wave keeps a ring of the next
// D k-steps in flight.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gather.hpp"  // u32x4

namespace spk {

constexpr int kMfmaNAlign = 16;  // N must be a multiple of this (one channel set)
constexpr int kMfmaK = 64;       // k per step: one mask word
constexpr int kMfmaSetStepBytes = 1024;  // one k-step of one channel set in the packed copy
constexpr int kMfmaMaxLds = 64 * 1024;   // LDS of one workgroup: partial tile + staged spike words

typedef int32_t mf_i32x4 __attribute__((ext_vector_type(4)));

constexpr int kBufferWordFormat = 0x00020000;  // buffer resource word 3: 32-bit data format (gfx9)

// Bytes of the packed copy of a K x N matrix.
inline int64_t mfma_packed_bytes(int64_t K, int64_t N) { return (K + kMfmaK - 1) / kMfmaK * kMfmaK * N; }

// The packed copy must be addressable by 31-bit byte offsets (one buffer
// resource) and N must split into whole channel sets.
inline bool mfma_supported(int64_t K, int64_t N)
{
    return N % kMfmaNAlign == 0 && mfma_packed_bytes(K, N) < (1ll << 31);
}

// LDS row pitch (in 64-bit words) of the staged spike words: odd, so that
// the 16 rows read by one operand load fall in distinct banks.
inline int mfma_stage_pitch(int wpr) { return wpr | 1; }

// One thread per 16-byte lane chunk of the packed copy.
constexpr int kPackBlock = 256;
__global__ __launch_bounds__(kPackBlock) void k_mfma_pack(const int8_t* __restrict__ W, int K, int N, int wpr,
                                                          int8_t* __restrict__ P, int64_t n_chunks)
{
    const int64_t id = (int64_t)blockIdx.x * kPackBlock + threadIdx.x;
    if (id >= n_chunks)
        return;
    const int l = (int)(id % 64);
    const int64_t s = (id / 64) % wpr;
    const int64_t t = id / (64 * (int64_t)wpr);
    const int64_t n = t * 16 + l % 16;
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

// Tile of a workgroup.  When the channel-set tiles divide evenly over the 8
// XCDs (workgroups are dispatched to them round-robin), the row tiles of one
// channel-set tile are all put on the same XCD.
__device__ inline void mfma_tile_of(int id, int n_rowtiles, int n_coltiles, int* ct, int* rt)
{
    if (n_coltiles % 8 == 0) {
        const int x = id % 8, i = id / 8;
        *ct = x + 8 * (i / n_rowtiles);
        *rt = i % n_rowtiles;
    } else {
        *ct = id / n_rowtiles;
        *rt = id % n_rowtiles;
    }
}

// Bytes of dynamic LDS of one workgroup: the partial-sum tile, then (unless
// the spike words are loaded directly) the staged spike words of its rows.
inline int mfma_lds_bytes(int RT, int CS, int wpr, bool direct = false)
{
    return RT * CS * 256 * (int)sizeof(int32_t) +
           (direct ? 0 : 16 * RT * mfma_stage_pitch(wpr) * (int)sizeof(uint64_t));
}

// One output tile (tile id `id` of the launch's n_rowtiles x n_coltiles
// tiles) of one projection.  DIRECT: instead of staging the tile's spike
// words in LDS behind a barrier, each lane loads the dword holding its 16
// bits of the step with that step's weights (for the smallest batches, where
// the staging round trip is a large share of a call and the extra loads find
// rows past B out of range, so they move no data).
template <int RT, int CS, int KW, int D, bool PRELOAD, bool ACC, bool DIRECT = false>
// Always inlined: as a called function it spills (the call ABI) and runs
// several times slower.
__device__ __attribute__((always_inline)) inline void mfma_tile(const int8_t* __restrict__ P, const float* __restrict__ scale, int N,
                                 const uint64_t* __restrict__ mask, int wpr, int B, int n_rowtiles, int n_coltiles,
                                 int id, float* __restrict__ out, int32_t* __restrict__ acc_out)
{
    constexpr int BLOCK = 64 * KW;
    constexpr int ROWS = 16 * RT;
    constexpr int RED = RT * CS * 256;  // INT32 entries of the partial-sum tile
    extern __shared__ __align__(16) uint8_t lds[];
    int32_t* red = reinterpret_cast<int32_t*>(lds);
    uint64_t* xs = reinterpret_cast<uint64_t*>(lds + RED * sizeof(int32_t));  // staged spike words (!DIRECT)
    const int pitch = wpr | 1;

    // wave index as a scalar, so that everything derived from it (k-steps,
    // buffer offsets) is known to be uniform across the wave
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int l = threadIdx.x % 64;
    const int q = l / 16;  // k-group of the operands, row group of the result
    const int c = l % 16;  // row of A, channel of B and of the result
    int ct, rt;
    mfma_tile_of(id, n_rowtiles, n_coltiles, &ct, &rt);
    const int m0 = rt * ROWS;
    const int t0 = ct * CS;  // first channel set of the tile

    // k-steps of this wave: wave, wave + KW, ...
    const int n_steps = (wpr - wave + KW - 1) / KW;

    // The weight copy is a buffer resource: the lane's offset is a fixed
    // vector register, the k-step a scalar, so addressing costs no vector ALU.
    const __amdgpu_buffer_rsrc_t prsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t*>(P), 0, (N / 16) * wpr * kMfmaSetStepBytes, kBufferWordFormat);
    // The mask is a buffer resource: rows at or past B read as 0.
    const __amdgpu_buffer_rsrc_t mrsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint64_t*>(mask), 0, B * wpr * (int)sizeof(uint64_t), kBufferWordFormat);
    // Weights of the wave's step i; DIRECT: also, per row subtile, the dword
    // holding bits 16q .. 16q + 15 of word s of row 16 ms + c.  A step past
    // the wave's last (the slots of a preload or ring deeper than the steps
    // left) is read at the end of the buffer: out of range, so the load
    // returns zeros and moves no data, where a re-read of the last step
    // would issue its requests again.  Those slots are never multiplied.
    const int w_records = (N / 16) * wpr * kMfmaSetStepBytes;
    const int m_records = B * wpr * (int)sizeof(uint64_t);
    auto load_w = [&](int i, u32x4 (&wv)[CS], uint32_t (&bv)[RT]) {
        const int s = wave + i * KW;
        const bool live = i < n_steps;
#pragma unroll
        for (int t = 0; t < CS; ++t)
            wv[t] = __builtin_amdgcn_raw_buffer_load_b128(
                prsrc, 16 * l, live ? ((t0 + t) * wpr + s) * kMfmaSetStepBytes : w_records, 0);
        if constexpr (DIRECT) {
#pragma unroll
            for (int ms = 0; ms < RT; ++ms)
                bv[ms] = __builtin_amdgcn_raw_buffer_load_b32(
                    mrsrc, live ? ((m0 + 16 * ms + c) * wpr + s) * (int)sizeof(uint64_t) + 4 * (q / 2) : m_records, 0,
                    0);
        }
    };

    // Output form (see the final loops).  Tall tiles (RT >= 4: batches of
    // more than 64 rows), where N and the output (and scale) addresses allow
    // it, write four consecutive channels of one row per thread with one
    // 16-byte store (quad e4 = entries 4 e4 .. 4 e4 + 3 of the partial tile);
    // otherwise one channel per thread and entry.  Either way the scales are
    // loaded now, so that the epilogue does not wait for them.
    constexpr int kPer = (RED + BLOCK - 1) / BLOCK;
    constexpr int kPer4 = (RED / 4 + BLOCK - 1) / BLOCK;
    const uintptr_t dst_addr = ACC ? reinterpret_cast<uintptr_t>(acc_out) : reinterpret_cast<uintptr_t>(out);
    const uintptr_t sc_addr = ACC ? 0 : reinterpret_cast<uintptr_t>(scale);
    const bool vec_out = RT >= 4 && N % 4 == 0 && ((dst_addr | sc_addr) & 15) == 0;
    f32x4 sc4[RT >= 4 ? kPer4 : 1];
    float sc[RT >= 4 ? 1 : kPer];
    if constexpr (!ACC) {
        if constexpr (RT >= 4) {
#pragma unroll
            for (int r = 0; r < kPer4; ++r) {
                const int e4 = threadIdx.x + r * BLOCK;
                const int t = (e4 / 64) % CS;
                sc4[r] = vec_out && e4 < RED / 4
                             ? *reinterpret_cast<const f32x4*>(scale + 16 * (t0 + t) + 4 * (e4 % 4))
                             : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
        } else {
#pragma unroll
            for (int r = 0; r < kPer; ++r) {
                const int e = threadIdx.x + r * BLOCK;
                const int t = (e / 256) % CS;
                sc[r] = e < RED ? scale[16 * (t0 + t) + e % 16] : 0.0f;
            }
        }
    }

    // Every wave has at least one k-step (the plan requires KW <= wpr).
    // Loads are unconditional (a step past the wave's last reads out of
    // range, see load_w): a conditional load would turn its registers into
    // phis that the compiler fills with copies.
    u32x4 wbuf[D][CS];
    uint32_t bbuf[D][RT];  // DIRECT: the spike dwords of each slot
#pragma unroll
    for (int d = 0; d < D; ++d)
        load_w(d, wbuf[d], bbuf[d]);

    // Stage the tile's spike words (ROWS rows x wpr words) unless DIRECT,
    // and zero the partial tile.
    if constexpr (DIRECT) {
        for (int e = threadIdx.x; e < RED; e += BLOCK)
            red[e] = 0;
    } else {
        const int total = ROWS * wpr;
        // loads in flight per thread before their stores: enough that a
        // tile of up to 128 words per row is staged in one round trip
        constexpr int kBatch = (ROWS * 128 + BLOCK - 1) / BLOCK < 4    ? 4
                               : (ROWS * 128 + BLOCK - 1) / BLOCK > 16 ? 16
                                                                        : (ROWS * 128 + BLOCK - 1) / BLOCK;
        for (int base = 0; base < total; base += kBatch * BLOCK) {
            u32x2 v[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int e = min(base + u * BLOCK + (int)threadIdx.x, total - 1);
                const int r = e / wpr, w = e - r * wpr;
                v[u] = __builtin_amdgcn_raw_buffer_load_b64(mrsrc, ((m0 + r) * wpr + w) * (int)sizeof(uint64_t), 0,
                                                            0);
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int e = base + u * BLOCK + (int)threadIdx.x;
                if (e < total) {
                    const int r = e / wpr, w = e - r * wpr;
                    xs[r * pitch + w] = __builtin_bit_cast(uint64_t, v[u]);
                }
            }
        }
        for (int e = threadIdx.x; e < RED; e += BLOCK)
            red[e] = 0;
        __syncthreads();
    }

    mf_i32x4 acc[RT][CS];
#pragma unroll
    for (int ms = 0; ms < RT; ++ms)
#pragma unroll
        for (int t = 0; t < CS; ++t)
            acc[ms][t] = mf_i32x4{0, 0, 0, 0};

    // Spikes 16q .. 16q + 15 of row 16 ms + c at the wave's step i (one
    // 16-bit LDS read per row subtile), and the A-operands built from them.
    const uint16_t* xs16 = reinterpret_cast<const uint16_t*>(xs);
    auto read_bits = [&](int i, uint32_t (&b)[RT]) {
        const int s = wave + i * KW;
#pragma unroll
        for (int ms = 0; ms < RT; ++ms)
            b[ms] = xs16[((16 * ms + c) * pitch + s) * 4 + q];
    };
    // DIRECT: this lane's 16 bits are the low or high half of its dword
    auto slot_bits = [&](const uint32_t (&bv)[RT], uint32_t (&b)[RT]) {
#pragma unroll
        for (int ms = 0; ms < RT; ++ms)
            b[ms] = bv[ms] >> (16 * (q & 1));
    };
    auto products = [&](const uint32_t (&b)[RT], const u32x4 (&wv)[CS]) {
        mf_i32x4 a[RT];
#pragma unroll
        for (int ms = 0; ms < RT; ++ms)
            a[ms] = mf_i32x4{(int32_t)expand_nibble(b[ms]), (int32_t)expand_nibble(b[ms] >> 4),
                             (int32_t)expand_nibble(b[ms] >> 8), (int32_t)expand_nibble(b[ms] >> 12)};
#pragma unroll
        for (int ms = 0; ms < RT; ++ms)
#pragma unroll
            for (int t = 0; t < CS; ++t)
                acc[ms][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ms], __builtin_bit_cast(mf_i32x4, wv[t]),
                                                                    acc[ms][t], 0, 0, 0);
    };

    if constexpr (PRELOAD) {
#pragma unroll
        for (int d = 0; d < D; ++d)
            if (d < n_steps) {
                uint32_t b[RT];
                if constexpr (DIRECT)
                    slot_bits(bbuf[d], b);
                else
                    read_bits(d, b);
                products(b, wbuf[d]);
            }
    } else if constexpr (DIRECT) {
        // Ring of D slots of weights and spike dwords; a slot is refilled
        // after its products with the step D ahead (out of range past the
        // wave's last step, as below).
        auto step = [&](int i, u32x4 (&wv)[CS], uint32_t (&bv)[RT], bool refill) {
            uint32_t b[RT];
            slot_bits(bv, b);
            products(b, wv);
            if (refill)
                load_w(i + D, wv, bv);
        };
        const int n_full = n_steps / D * D;
        int i0 = 0;
        for (; i0 < n_full; i0 += D) {
#pragma unroll
            for (int d = 0; d < D; ++d)
                step(i0 + d, wbuf[d], bbuf[d], true);
        }
#pragma unroll
        for (int d = 0; d < D; ++d)
            if (i0 + d < n_steps)
                step(i0 + d, wbuf[d], bbuf[d], false);
    } else {
        // Ring of D slots; the loop is unrolled by D so slot indices stay
        // static.  A slot is refilled after its products (the load then
        // has D - 1 steps of cover) with the step D ahead, read out of range
        // past the wave's last step: an unconditional load keeps the slot
        // out of phi copies, and the extra loads move no data.  The spike
        // bits of the next step are read from LDS one step ahead, so their
        // latency hides behind the current step's products.
        uint32_t bits[RT];
        read_bits(0, bits);
        auto step = [&](int i, u32x4 (&wv)[CS], uint32_t (&bv)[RT], bool refill) {
            uint32_t nb[RT];
            read_bits(min(i + 1, n_steps - 1), nb);
            products(bits, wv);
            if (refill)
                load_w(i + D, wv, bv);
#pragma unroll
            for (int ms = 0; ms < RT; ++ms)
                bits[ms] = nb[ms];
        };
        const int n_full = n_steps / D * D;
        int i0 = 0;
        for (; i0 < n_full; i0 += D) {
#pragma unroll
            for (int d = 0; d < D; ++d)
                step(i0 + d, wbuf[d], bbuf[d], true);
        }
#pragma unroll
        for (int d = 0; d < D; ++d)
            if (i0 + d < n_steps)
                step(i0 + d, wbuf[d], bbuf[d], false);
    }
    if constexpr (DIRECT)
        __syncthreads();  // the partial tile is zeroed before any wave adds to it

    // Partial tiles of the waves -> LDS (integer atomics: order-free).
    // Entry ((ms * CS + t) * 4 + j) * 64 + lane holds register j of lane
    // `lane` of accumulator (ms, t).
#pragma unroll
    for (int ms = 0; ms < RT; ++ms)
#pragma unroll
        for (int t = 0; t < CS; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                atomicAdd(&red[((ms * CS + t) * 4 + j) * 64 + l], acc[ms][t][j]);
    __syncthreads();

    // entry e -> row m0 + 16 ms + 4 (lane / 16) + j, channel 16 (t0 + t) + lane % 16
    if constexpr (RT >= 4) if (vec_out) {
        // quad e4 -> entries 4 e4 .. 4 e4 + 3: block g = e4 / 16 of 64
        // entries, lanes 4 (e4 % 16) .. + 3, i.e. one row, four channels
#pragma unroll
        for (int r = 0; r < kPer4; ++r) {
            const int e4 = threadIdx.x + r * BLOCK;
            if (e4 >= RED / 4)
                break;
            const int g = e4 / 16, qd = e4 % 16;
            const int j = g % 4, mt = g / 4;
            const int ms = mt / CS, t = mt % CS;
            const int b = m0 + 16 * ms + 4 * (qd / 4) + j;
            if (b >= B)
                continue;
            const int64_t n0 = 16 * (t0 + t) + 4 * (qd % 4);
            const i32x4 sum = *reinterpret_cast<const i32x4*>(red + 4 * e4);
            if constexpr (ACC) {
                *reinterpret_cast<i32x4*>(acc_out + (int64_t)b * N + n0) = sum;
            } else {
                const f32x4 s4 = sc4[r];
                f32x4 y;  // exact for |sum| < 2^24, RNE beyond; one binary32 multiply each
                y.x = (float)sum.x * s4.x;
                y.y = (float)sum.y * s4.y;
                y.z = (float)sum.z * s4.z;
                y.w = (float)sum.w * s4.w;
                __builtin_nontemporal_store(y, reinterpret_cast<f32x4*>(out + (int64_t)b * N + n0));
            }
        }
        return;
    }
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
        const int e = threadIdx.x + r * BLOCK;
        if (e >= RED)
            break;
        const int lane = e % 64, g = e / 64;
        const int j = g % 4, mt = g / 4;
        const int ms = mt / CS, t = mt % CS;
        const int b = m0 + 16 * ms + 4 * (lane / 16) + j;
        if (b >= B)
            continue;
        const int64_t n = 16 * (t0 + t) + lane % 16;
        const int32_t sum = red[e];
        if constexpr (ACC) {
            acc_out[(int64_t)b * N + n] = sum;
        } else {
            const float as_float = (float)sum;  // exact for |sum| < 2^24, RNE beyond
            out[(int64_t)b * N + n] = as_float * (RT >= 4 ? scale[n] : sc[RT >= 4 ? 0 : r]);
        }
    }
}

template <int RT, int CS, int KW, int D, bool PRELOAD, bool ACC, bool DIRECT>
__global__ __launch_bounds__(64 * KW) void k_mfma(const int8_t* __restrict__ P, const float* __restrict__ scale,
                                                  int N, const uint64_t* __restrict__ mask, int wpr, int B,
                                                  int n_rowtiles, int n_coltiles, float* __restrict__ out,
                                                  int32_t* __restrict__ acc_out)
{
    mfma_tile<RT, CS, KW, D, PRELOAD, ACC, DIRECT>(P, scale, N, mask, wpr, B, n_rowtiles, n_coltiles, blockIdx.x,
                                                   out, acc_out);
}

// Several projections of B given spike rows each, in one launch: item j
// (packed weights P[j], scales, K_j) reads its rows at word mask_off[j] of
// the mask buffer and writes its outputs at float out_off[j].  Every item
// has the same N and B, so the same tile count; workgroup b runs tile
// b % tiles of item b / tiles.  (Tiles per item are a multiple of 8 when
// the channel tiles are, so the XCD grouping of mfma_tile_of holds per
// item.)  The ring form serves any k-step count.
constexpr int kMfmaMaxItems = 64;
struct MfmaItems {
    const int8_t* P[kMfmaMaxItems];
    const float* scale[kMfmaMaxItems];
    int64_t mask_off[kMfmaMaxItems];
    int64_t out_off[kMfmaMaxItems];
    int32_t wpr[kMfmaMaxItems];
};

template <int RT, int CS, int KW, int D>
__global__ __launch_bounds__(64 * KW) void k_mfma_items(const MfmaItems items, int N, const uint64_t* __restrict__ mask,
                                                        int B, int n_rowtiles, int n_coltiles, float* __restrict__ out)
{
    const int tiles = n_rowtiles * n_coltiles;
    const int item = blockIdx.x / tiles;
    const int id = blockIdx.x - item * tiles;
    mfma_tile<RT, CS, KW, D, false, false>(items.P[item], items.scale[item], N, mask + items.mask_off[item],
                                           items.wpr[item], B, n_rowtiles, n_coltiles, id, out + items.out_off[item],
                                           nullptr);
}

// Launch configuration of the matrix-core path.
struct MfmaPlan {
    int rt, cs, kw, d;
    bool preload;
    bool direct = false;  // spike words loaded per k-step instead of staged in LDS
};

// Batches up to this many rows load their spike words directly (measured:
// a batch-1 stack of 44 dependent calls on cold weights takes 184 us with
// direct loads against 196 us staged; from 8 rows on, staging wins).
constexpr int kMfmaDirectMaxB = 4;

// Instantiated plans.  Every plan needs KW <= wpr (each wave has at least
// one k-step); PRELOAD plans also need every wave's k-step count to be at
// most D.
#define SPK_MFMA_PLANS(X)                                                                                          \
    X(1, 1, 1, 4, true) X(1, 1, 2, 4, true) X(1, 1, 4, 4, true) X(1, 1, 4, 8, true) X(1, 1, 8, 4, true)           \
    X(1, 1, 8, 8, true) X(1, 1, 8, 12, true) X(1, 1, 16, 4, true) X(1, 1, 16, 8, true) X(1, 2, 4, 4, true)       \
    X(1, 2, 4, 8, true) X(1, 2, 8, 4, true) X(1, 2, 8, 8, true) X(1, 2, 8, 12, true) X(1, 2, 16, 4, true)        \
    X(1, 2, 16, 8, true) X(2, 1, 4, 8, true) X(2, 1, 8, 4, true) X(2, 1, 8, 8, true) X(2, 1, 8, 12, true)        \
    X(2, 1, 16, 8, true) X(2, 2, 8, 8, true) X(2, 2, 8, 12, true) X(4, 1, 1, 4, true) X(4, 1, 2, 4, true)        \
    X(4, 1, 2, 8, true) X(4, 1, 4, 4, true) X(4, 1, 4, 8, true) X(4, 1, 8, 12, true) X(4, 1, 16, 8, true)        \
    X(1, 1, 8, 4, false) X(1, 2, 8, 4, false) X(1, 3, 8, 4, false) X(2, 1, 8, 4, false) X(2, 2, 8, 4, false)     \
    X(2, 3, 8, 4, false) X(4, 1, 8, 4, false) X(4, 2, 8, 4, false) X(4, 3, 8, 4, false) X(1, 1, 16, 4, false)    \
    X(4, 3, 8, 2, false) X(4, 4, 8, 2, false) X(4, 4, 8, 4, false) X(4, 3, 4, 4, false) X(8, 3, 8, 2, false)     \
    X(8, 2, 8, 4, false) X(4, 6, 8, 2, false) X(4, 3, 16, 2, false) X(4, 3, 16, 4, false) X(4, 2, 16, 4, false)  \
    X(2, 3, 16, 4, false) X(1, 2, 1, 4, true) X(1, 2, 2, 4, true) X(1, 2, 16, 4, false) X(1, 1, 16, 2, false)    \
    X(1, 2, 16, 2, false) X(1, 3, 16, 2, false) X(2, 1, 16, 2, false) X(2, 2, 16, 2, false) X(2, 3, 16, 2, false) \
    X(4, 1, 16, 2, false) X(4, 2, 16, 2, false) X(1, 1, 1, 4, false) X(1, 2, 1, 4, false) X(1, 1, 2, 4, false)    \
    X(1, 2, 2, 4, false) X(1, 1, 4, 4, false) X(1, 2, 4, 4, false) X(4, 1, 1, 2, false) X(4, 3, 1, 2, false)     \
    X(4, 1, 2, 2, false) X(4, 3, 2, 2, false)

// Plans also instantiated with direct spike loads: the automatic plans of
// batches up to kMfmaDirectMaxB rows (one 16-row subtile and one channel set
// per workgroup; every k-step preloaded up to 6 steps per wave, i.e. for
// K <= 6144, a ring of 2 beyond; with 8 waves the preload depth equals the
// wave's step count, so no wave issues a duplicate load).
#define SPK_MFMA_DIRECT_PLANS(X) \
    X(1, 1, 1, 4, true) X(1, 1, 2, 4, true) X(1, 1, 4, 4, true) X(1, 1, 8, 4, true) X(1, 1, 16, 2, false) \
    X(1, 1, 16, 6, true) X(1, 1, 8, 1, true) X(1, 1, 8, 2, true) X(1, 1, 8, 3, true)

inline bool mfma_instantiated(const MfmaPlan& p)
{
    bool found = false;
#define SPK_FIND(RT, CS, KW, D, PRE) \
    found = found || (p.rt == RT && p.cs == CS && p.kw == KW && p.d == D && p.preload == PRE);
    if (p.direct) {
        SPK_MFMA_DIRECT_PLANS(SPK_FIND)
    } else {
        SPK_MFMA_PLANS(SPK_FIND)
    }
#undef SPK_FIND
    return found;
}

// Plan for B rows (automatic unless overridden: a field > 0 fixes it).
// Small batches (B <= 64): 16-row by 16-channel tiles, enough waves that
// every wave's k-steps are all in flight at once.  Large batches: 64-row
// tiles (fewer if the staged spike words would not fit) by 48, 32 or 16
// channels, 8 waves with 4 k-steps in flight each.
inline MfmaPlan mfma_plan(int K, int N, int B, int rt_req, int cs_req, int kw_req, int d_req)
{
    const int wpr = (K + 63) / 64;
    const int sets = N / 16;
    MfmaPlan p{};
    if (B <= 16) {
        // one row tile: one channel set per workgroup (the most workgroups),
        // 8 waves for short K, 16 for long K (measured per dependent call on
        // the 1536- and 6144-input shapes)
        p.rt = 1;
        p.cs = 1;
        p.kw = wpr <= 32 ? 8 : 16;
    } else if (B <= 64) {
        // measured on the 64-row decode stack: two channel sets, 8 waves
        p.rt = 1;
        p.cs = sets % 2 == 0 ? 2 : 1;
        p.kw = wpr <= 128 ? 8 : 16;
    } else if (wpr < 32) {
        p.rt = 4;
        p.cs = 1;
        p.kw = 4;
    } else {
        // measured on the 512-token prefill: 64 rows x 48 channels, 16 waves
        p.rt = 4;
        p.cs = sets % 3 == 0 ? 3 : sets % 2 == 0 ? 2 : 1;
        p.kw = 16;
    }
    while (p.kw > 1 && p.kw > wpr)  // every wave needs a k-step
        p.kw /= 2;
    if (rt_req > 0)
        p.rt = rt_req;
    if (cs_req > 0)
        p.cs = cs_req;
    if (kw_req > 0)
        p.kw = kw_req;
    const int steps = (wpr + p.kw - 1) / p.kw;
    if (d_req > 0)
        p.d = d_req;
    else if (B <= 16)
        // short K: every step preloaded; long K: a ring of 2, except that
        // batches of up to kMfmaDirectMaxB rows (direct spike loads) preload
        // up to 6 steps per wave: one memory round trip on cold weights
        // (measured on the cold 44-projection batch-1 chain: 181 us per
        // token against 185 us with the ring, 192 us with a depth of 8)
        p.d = wpr <= 32 ? 4 : B <= kMfmaDirectMaxB && steps <= 6 ? 6 : 2;
    else if (B <= 64)
        p.d = 4;  // preloads up to 4 steps per wave, a ring of 4 beyond
    else if (wpr < 32)
        p.d = steps <= 4 ? 4 : 8;
    else
        p.d = 2;
    // small batches preload every k-step where they fit; large batches keep
    // a ring (which also serves waves with fewer steps than its depth)
    p.preload = (B <= 64 || wpr < 32 || d_req > 0) && steps <= p.d;
    if (rt_req <= 0) {
        // the staged words of the tile's rows must fit the LDS budget
        while (p.rt > 1 && mfma_lds_bytes(p.rt, p.cs, wpr) > kMfmaMaxLds)
            p.rt /= 2;
    }
    // a ring kernel runs any step count: use it where the preloading
    // variant of a tuned combination is not instantiated
    if (p.preload && !mfma_instantiated(p)) {
        MfmaPlan r = p;
        r.preload = false;
        if (mfma_instantiated(r))
            p = r;
    }
    // the smallest batches load their spike words directly where that
    // variant of the plan exists
    if (B <= kMfmaDirectMaxB) {
        MfmaPlan r = p;
        r.direct = true;
        if (d_req <= 0 && r.preload) {
            // a depth equal to the step count: a deeper preload re-issues the
            // last step's loads, which costs a cold call about 0.2 us
            // (measured on the 44-projection batch-1 chain: 174 us per token
            // with 3 steps at depth 3 against 179 us at depth 4)
            MfmaPlan e = r;
            e.d = (wpr + e.kw - 1) / e.kw;
            if (mfma_instantiated(e))
                r = e;
        }
        if (mfma_instantiated(r))
            p = r;
    }
    return p;
}

// A ring plan (any k-step count) for a launch whose projections all have
// at least min_wpr k-steps: an instantiated ring plan with a channel-set
// count dividing N / 16 and at most min_wpr waves, preferring p's row tile,
// then p's channel sets, then the most waves up to p's, then p's depth.
// Returns false if none.
inline bool mfma_ring_plan(MfmaPlan& p, int min_wpr, int N)
{
    const int sets = N / 16;
    MfmaPlan best{};
    int best_score = -1;
#define SPK_RING(RT, CS, KW, D, PRE)                                                                 \
    if (!PRE && KW <= min_wpr && sets % CS == 0) {                                                  \
        const int score = (RT == p.rt ? 1 << 24 : 0) + (CS == p.cs ? 1 << 20 : 0) +                 \
                          (KW <= p.kw ? KW << 8 : 0) + (D == p.d ? 1 : 0);                          \
        if (score > best_score) {                                                                    \
            best_score = score;                                                                      \
            best = MfmaPlan{RT, CS, KW, D, false};                                                   \
        }                                                                                            \
    }
    SPK_MFMA_PLANS(SPK_RING)
#undef SPK_RING
    if (best_score < 0)
        return false;
    p = best;
    return true;
}

// Plan code reported by the library: rt | cs << 4 | kw << 8 | d << 16 |
// preload << 24 | direct << 25.
inline int mfma_plan_code(const MfmaPlan& p)
{
    return p.rt | p.cs << 4 | p.kw << 8 | p.d << 16 | (p.preload ? 1 << 24 : 0) | (p.direct ? 1 << 25 : 0);
}

template <int RT, int CS, int KW, int D, bool PRELOAD, bool DIRECT>
hipError_t launch_mfma_t(const int8_t* P, const float* scale, int K, int N, const uint64_t* mask, int B,
                         float* out, int32_t* acc, bool want_acc, hipStream_t st)
{
    const int wpr = (K + 63) / 64;
    const int n_coltiles = N / (16 * CS);
    const int n_rowtiles = (B + 16 * RT - 1) / (16 * RT);
    const int64_t units = (int64_t)n_coltiles * n_rowtiles;
    const int lds = mfma_lds_bytes(RT, CS, wpr, DIRECT);
    if (units > 0x7fffffff)
        return hipErrorInvalidValue;
    if (want_acc)
        hipLaunchKernelGGL((k_mfma<RT, CS, KW, D, PRELOAD, true, DIRECT>), dim3((unsigned)units), dim3(64 * KW), lds,
                           st, P, scale, N, mask, wpr, B, n_rowtiles, n_coltiles, out, acc);
    else
        hipLaunchKernelGGL((k_mfma<RT, CS, KW, D, PRELOAD, false, DIRECT>), dim3((unsigned)units), dim3(64 * KW),
                           lds, st, P, scale, N, mask, wpr, B, n_rowtiles, n_coltiles, out, acc);
    return hipGetLastError();
}

template <int RT, int CS, int KW, int D>
hipError_t launch_mfma_items_t(const MfmaItems& items, int n_items, int max_wpr, int N, const uint64_t* mask, int B,
                               float* out, hipStream_t st)
{
    const int n_coltiles = N / (16 * CS);
    const int n_rowtiles = (B + 16 * RT - 1) / (16 * RT);
    const int64_t units = (int64_t)n_coltiles * n_rowtiles * n_items;
    if (units > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_items<RT, CS, KW, D>), dim3((unsigned)units), dim3(64 * KW),
                       mfma_lds_bytes(RT, CS, max_wpr), st, items, N, mask, B, n_rowtiles, n_coltiles, out);
    return hipGetLastError();
}

// Launch of several projections for a ring plan (p.preload must be false).
inline hipError_t launch_mfma_items(const MfmaPlan& p, const MfmaItems& items, int n_items, int max_wpr, int N,
                                    const uint64_t* mask, int B, float* out, hipStream_t st)
{
#define SPK_LAUNCH_ITEMS(RT, CS, KW, D, PRE)                                                       \
    if (!PRE && p.rt == RT && p.cs == CS && p.kw == KW && p.d == D && !p.preload)              \
        return launch_mfma_items_t<RT, CS, KW, D>(items, n_items, max_wpr, N, mask, B, out, st);
    SPK_MFMA_PLANS(SPK_LAUNCH_ITEMS)
#undef SPK_LAUNCH_ITEMS
    return hipErrorInvalidValue;
}

// Codes of every instantiated plan (host memory, up to cap); returns the count.
inline int mfma_plan_codes(int32_t* codes, int cap)
{
    int n = 0;
#define SPK_CODE(RT, CS, KW, D, PRE)                                      \
    if (codes && n < cap)                                                  \
        codes[n] = mfma_plan_code(MfmaPlan{RT, CS, KW, D, PRE, false});    \
    ++n;
    SPK_MFMA_PLANS(SPK_CODE)
#undef SPK_CODE
#define SPK_CODE_DIRECT(RT, CS, KW, D, PRE)                               \
    if (codes && n < cap)                                                  \
        codes[n] = mfma_plan_code(MfmaPlan{RT, CS, KW, D, PRE, true});     \
    ++n;
    SPK_MFMA_DIRECT_PLANS(SPK_CODE_DIRECT)
#undef SPK_CODE_DIRECT
    return n;
}

// Is the plan instantiated and runnable for this shape?  Returns 0 or a
// message.
inline const char* mfma_plan_check(const MfmaPlan& p, int K, int N)
{
    const int wpr = (K + 63) / 64;
    if (!mfma_instantiated(p))
        return "this (row tile, channel sets, waves, depth) combination is not instantiated";
    if ((N / 16) % p.cs != 0)
        return "N / 16 is not a multiple of the tile's channel sets";
    if (mfma_lds_bytes(p.rt, p.cs, wpr) > kMfmaMaxLds)
        return "the tile's staged spike words exceed the LDS budget";
    if (wpr < p.kw)
        return "fewer k-steps than waves";
    if (p.preload && (wpr + p.kw - 1) / p.kw > p.d)
        return "more k-steps per wave than the preload depth";
    return nullptr;
}

inline hipError_t launch_mfma(const MfmaPlan& p, const int8_t* P, const float* scale, int K, int N,
                              const uint64_t* mask, int B, float* out, int32_t* acc, bool want_acc, hipStream_t st)
{
#define SPK_LAUNCH(RT, CS, KW, D, PRE)                                                              \
    if (p.rt == RT && p.cs == CS && p.kw == KW && p.d == D && p.preload == PRE)                  \
        return launch_mfma_t<RT, CS, KW, D, PRE, false>(P, scale, K, N, mask, B, out, acc, want_acc, st);
#define SPK_LAUNCH_DIRECT(RT, CS, KW, D, PRE)                                                       \
    if (p.rt == RT && p.cs == CS && p.kw == KW && p.d == D && p.preload == PRE)                  \
        return launch_mfma_t<RT, CS, KW, D, PRE, true>(P, scale, K, N, mask, B, out, acc, want_acc, st);
    if (p.direct) {
        SPK_MFMA_DIRECT_PLANS(SPK_LAUNCH_DIRECT)
    } else {
        SPK_MFMA_PLANS(SPK_LAUNCH)
    }
#undef SPK_LAUNCH
#undef SPK_LAUNCH_DIRECT
    return hipErrorInvalidValue;
}

}  // namespace spk
