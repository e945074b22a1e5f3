// Active-column gather for the spike-gated INT8 projection on CDNA4 (gfx950).
//
// Computes Eq. (sparse) of the paper (Sec. 2.3): for a binary spike row x,
// y[n] = scale[n] * sum_{k in A} Q[n][k] with A = {k : x_k = 1} (Sec. 2.2).
// Weights are column-major (W[k*N + n]), so each active column is one
// contiguous run of N bytes; inactive columns are never read.
//
// One workgroup ("unit") owns a range of output-channel tiles and a slice of
// the K axis for one spike row:
//   1. compaction: the slice's mask words become an ascending list of active
//      column indices in LDS (popcount + wavefront prefix scan, then every
//      thread writes the set bits of its own words at its prefix offset);
//   2. gather: lane groups walk the list; every lane streams V bytes of each
//      active column (one coalesced load per column) and adds the
//      sign-extended bytes into V INT32 registers.  Each lane keeps a ring of
//      U load slots: a slot is added and at once refilled with the column U
//      steps ahead, so U columns stay in flight; loads are unconditional
//      buffer loads, and positions past the list read as zero (out-of-range
//      offset), so no register copies or branches stall the ring;
//   3. the lane groups of a wave are summed with cross-lane shuffles, the
//      waves' partial sums in LDS;
//   4. a single-slice unit converts and scales directly; with several
//      K-slices, partials are folded into an INT32 workspace with device-
//      scope atomic adds (exact, so order-independent), and the last unit of
//      the tile to arrive (atomic completion counter) reads the totals back
//      with atomic exchange -- which also re-zeroes the workspace -- and
//      writes fl32(fl32(acc) * scale[n]).  The counter is reset too, so the
//      next call on the same stream starts from a clean workspace.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "buffer.hpp"

namespace spk {

constexpr int kMaxSliceWords = 256;  // mask words per K-slice (16384 columns)

template <int BLOCK>
struct SliceLds {
    static_assert(BLOCK % 64 == 0 && BLOCK >= 64 && BLOCK <= 1024, "block must be whole waves");
    static constexpr int kWaves = BLOCK / 64;
    int32_t wave_total[kWaves];
    int32_t is_last;
};

// Mask words of one thread: words [w0 + t * per, w0 + t * per + per) of the
// slice [w0, w0 + nw), per = ceil(nw / BLOCK) <= kPer, with the bits at or
// above K cleared (padding).  Words past the slice are zero.
template <int BLOCK>
struct ThreadWords {
    static constexpr int kPer = (kMaxSliceWords + BLOCK - 1) / BLOCK;
    uint64_t w[kPer];
};

template <int BLOCK>
__device__ inline void load_words(const uint64_t* __restrict__ row, int w0, int nw, int K, ThreadWords<BLOCK>& tw)
{
    const int per = (nw + BLOCK - 1) / BLOCK;
    const int first = threadIdx.x * per;
#pragma unroll
    for (int i = 0; i < ThreadWords<BLOCK>::kPer; ++i) {
        const int j = first + i;
        uint64_t word = 0;
        if (i < per && j < nw) {
            const int w = w0 + j;
            word = row[w];
            const int valid = K - 64 * w;  // bits of this word below K
            if (valid < 64)
                word &= valid <= 0 ? 0ull : ((1ull << valid) - 1ull);
        }
        tw.w[i] = word;
    }
}

// Active positions of the slice whose words the threads hold, ascending:
// emit(pos, k_rel) is called once per active bit with its rank pos in the
// list and its index k_rel relative to bit 64*w0.  Returns |A| of the slice
// in every thread.  Each thread owns a contiguous run of words, so the scan
// over threads is a scan in word order; every thread emits the set bits of
// its own words.  Two workgroup barriers.
template <int BLOCK, class Emit>
__device__ inline int compact_words(const ThreadWords<BLOCK>& tw, int nw, SliceLds<BLOCK>& s, Emit emit)
{
    constexpr int kWaves = SliceLds<BLOCK>::kWaves;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int per = (nw + BLOCK - 1) / BLOCK;
    const int first = t * per;
    int pc = 0;
#pragma unroll
    for (int i = 0; i < ThreadWords<BLOCK>::kPer; ++i)
        pc += __popcll(tw.w[i]);
    int incl = pc;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int up = __shfl_up(incl, d, 64);
        if (lane >= d)
            incl += up;
    }
    if (lane == 63)
        s.wave_total[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
        const int wt = s.wave_total[v];
        before += v < wave ? wt : 0;
        total += wt;
    }
    int pos = before + incl - pc;  // exclusive prefix of this thread's words
#pragma unroll
    for (int i = 0; i < ThreadWords<BLOCK>::kPer; ++i) {
        uint64_t word = tw.w[i];
        const int kb = 64 * (first + i);
        while (word) {
            emit(pos++, kb + (int)__builtin_ctzll(word));
            word &= word - 1ull;
        }
    }
    __syncthreads();
    return total;
}

// Active positions of mask words [w0, w0 + nw) of one row (load_words, then
// compact_words).  Requires nw <= kMaxSliceWords.
template <int BLOCK, class Emit>
__device__ inline int compact_slice(const uint64_t* __restrict__ row, int w0, int nw, int K, SliceLds<BLOCK>& s,
                                    Emit emit)
{
    ThreadWords<BLOCK> tw;
    load_words<BLOCK>(row, w0, nw, K, tw);
    return compact_words<BLOCK>(tw, nw, s, emit);
}

// Cross-workgroup hand-off without cache maintenance.  A device-scope
// release/acquire fence on this chip writes back and invalidates the whole
// L2 of the XCD (buffer_wbl2 / buffer_inv), which stalls every workgroup that
// shares it.  The split-K hand-offs here need none of that: every datum that
// crosses workgroups is written and read with device-coherent operations
// (INT32 atomics, or atomic stores/loads of device scope, which bypass the
// non-coherent caches), so it is enough that a workgroup's writes have
// completed -- s_waitcnt 0 waits until the memory system has acknowledged
// them -- before the completion counter is bumped, and that the last
// workgroup reads only after it has seen the counter.
__device__ inline void wait_writes_done() { __builtin_amdgcn_s_waitcnt(0); }

// V bytes of one column for one lane, added into V INT32 accumulators.
// NT loads carry the nontemporal hint (streamed weights are not re-read).
template <class T, bool NT>
__device__ inline T load_hint(const T* p)
{
    if constexpr (NT)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}

template <int V, bool NT>
struct Chunk;

// acc[i] += sign-extended byte i of d: one VALU op per byte, an SDWA add
// whose first operand selects and sign-extends the byte (the compiler's own
// lowering takes a bit-field extract per byte plus three-operand adds).
__device__ inline void add_i8x4(int32_t* acc, uint32_t d)
{
    asm("v_add_u32_sdwa %0, sext(%1), %0 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 src1_sel:DWORD"
        : "+v"(acc[0]) : "v"(d));
    asm("v_add_u32_sdwa %0, sext(%1), %0 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD"
        : "+v"(acc[1]) : "v"(d));
    asm("v_add_u32_sdwa %0, sext(%1), %0 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:DWORD"
        : "+v"(acc[2]) : "v"(d));
    asm("v_add_u32_sdwa %0, sext(%1), %0 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 src1_sel:DWORD"
        : "+v"(acc[3]) : "v"(d));
}

template <bool NT>
struct Chunk<16, NT> {
    u32x4 v;
    __device__ void load(const int8_t* p) { v = load_hint<u32x4, NT>(reinterpret_cast<const u32x4*>(p)); }
    __device__ void zero() { v = u32x4{0, 0, 0, 0}; }
    __device__ void add(int32_t* acc) const
    {
        add_i8x4(acc + 0, v.x);
        add_i8x4(acc + 4, v.y);
        add_i8x4(acc + 8, v.z);
        add_i8x4(acc + 12, v.w);
    }
};
template <bool NT>
struct Chunk<8, NT> {
    u32x2 v;
    __device__ void load(const int8_t* p) { v = load_hint<u32x2, NT>(reinterpret_cast<const u32x2*>(p)); }
    __device__ void zero() { v = u32x2{0, 0}; }
    __device__ void add(int32_t* acc) const
    {
        add_i8x4(acc + 0, v.x);
        add_i8x4(acc + 4, v.y);
    }
};
template <bool NT>
struct Chunk<4, NT> {
    uint32_t v;
    __device__ void load(const int8_t* p) { v = load_hint<uint32_t, NT>(reinterpret_cast<const uint32_t*>(p)); }
    __device__ void zero() { v = 0; }
    __device__ void add(int32_t* acc) const { add_i8x4(acc, v); }
};
template <bool NT>
struct Chunk<1, NT> {  // any N, any alignment
    int8_t v;
    __device__ void load(const int8_t* p) { v = *p; }
    __device__ void zero() { v = 0; }
    __device__ void add(int32_t* acc) const { acc[0] += (int32_t)v; }
};

// The same loads through a buffer resource (buffer.hpp): offsets past the
// resource read as zero.  NT sets the nontemporal cache policy.

template <int V, bool NT>
struct BufChunk;
// Exact lower-width partial sums (paper Sec. 2.3: bounded active counts may
// sum in fewer bits).  Two channels share a 32-bit register as 16-bit
// halves holding biased sums: byte b enters as b + 128 in [0, 255], so up
// to 257 columns sum without overflow, and the bias is removed when the
// halves are added into the INT32 totals (every at most kI16MaxAdds
// columns).  Per four weight bytes: one XOR, two byte permutes and two
// packed 16-bit adds.
constexpr int kI16MaxAdds = 256;
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// even += (byte 0, byte 2) and odd += (byte 1, byte 3) of d, biased.
__device__ inline void add_i8x4_i16(uint32_t& even, uint32_t& odd, uint32_t d)
{
    const uint32_t u = d ^ 0x80808080u;
    const uint32_t e = __builtin_amdgcn_perm(0u, u, 0x0c020c00u);  // bytes 0 and 2 into the two halves
    const uint32_t o = __builtin_amdgcn_perm(0u, u, 0x0c030c01u);  // bytes 1 and 3
    even = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, even) + __builtin_bit_cast(u16x2, e));
    odd = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, odd) + __builtin_bit_cast(u16x2, o));
}

// acc[4i + 0, 2] and acc[4i + 1, 3] take the halves of p[2i] and p[2i + 1]
// less the bias of n adds; p is cleared.
__device__ inline void flush_i16(int32_t (&acc)[16], uint32_t (&p)[8], int n)
{
    const int32_t bias = 128 * n;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        acc[4 * i + 0] += (int32_t)(p[2 * i] & 0xffffu) - bias;
        acc[4 * i + 2] += (int32_t)(p[2 * i] >> 16) - bias;
        acc[4 * i + 1] += (int32_t)(p[2 * i + 1] & 0xffffu) - bias;
        acc[4 * i + 3] += (int32_t)(p[2 * i + 1] >> 16) - bias;
        p[2 * i] = 0;
        p[2 * i + 1] = 0;
    }
}

template <bool NT>
struct BufChunk<16, NT> {
    u32x4 v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, NT ? 2 : 0); }
    __device__ void add(int32_t* acc) const
    {
        add_i8x4(acc + 0, v.x);
        add_i8x4(acc + 4, v.y);
        add_i8x4(acc + 8, v.z);
        add_i8x4(acc + 12, v.w);
    }
    __device__ void add_i16(uint32_t (&p)[8]) const
    {
        add_i8x4_i16(p[0], p[1], v.x);
        add_i8x4_i16(p[2], p[3], v.y);
        add_i8x4_i16(p[4], p[5], v.z);
        add_i8x4_i16(p[6], p[7], v.w);
    }
};
template <bool NT>
struct BufChunk<8, NT> {
    u32x2 v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, NT ? 2 : 0); }
    __device__ void add(int32_t* acc) const
    {
        add_i8x4(acc + 0, v.x);
        add_i8x4(acc + 4, v.y);
    }
};
template <bool NT>
struct BufChunk<4, NT> {
    uint32_t v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, NT ? 2 : 0); }
    __device__ void add(int32_t* acc) const { add_i8x4(acc, v); }
};
template <bool NT>
struct BufChunk<1, NT> {
    uint8_t v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b8(r, off, 0, NT ? 2 : 0); }
    __device__ void add(int32_t* acc) const { acc[0] += (int32_t)(int8_t)v; }
};

// Launch shape.  Lane groups of LG lanes (a group may span waves); a lane
// covers V consecutive output channels, a group one tile of TB = LG * V
// channels of one column at a time; U columns per group are in flight;
// BLOCK threads per workgroup; NT marks weight loads nontemporal; I16 sums
// in exact 16-bit partials (V = 16, buffer-resource kernels).
template <int V_, int LG_, int U_, int BLOCK_, bool NT_ = false, bool I16_ = false>
struct Shape {
    static constexpr int V = V_, LG = LG_, U = U_, BLOCK = BLOCK_;
    static constexpr bool NT = NT_;
    static constexpr bool I16 = I16_;
    static_assert(!I16 || (V == 16 && kI16MaxAdds % U == 0), "16-bit partials: 16 channels per lane");
    static constexpr int kTile = V * LG;
    static constexpr int kGroups = BLOCK / LG;
    static_assert(BLOCK % LG == 0 && LG >= 1 && LG <= 64 && 64 % LG == 0, "lane groups must tile a wave");
    static_assert(U >= 1 && U <= 16, "unroll");
};

// Sum the active columns listed in `list` (indices relative to kbase) over
// this lane's V channels starting at byte n_lane of each column.
template <class S>
__device__ inline void gather_columns(const int8_t* __restrict__ W, int64_t N, int64_t kbase, int64_t n_lane,
                                      bool lane_in_range, const uint16_t* list, int cnt, int32_t (&acc)[S::V])
{
    constexpr int G = S::kGroups;
    constexpr int U = S::U;
#pragma unroll
    for (int j = 0; j < S::V; ++j)
        acc[j] = 0;
    if (!lane_in_range)
        return;
    const int8_t* base = W + n_lane;
    int i = threadIdx.x / S::LG;
    if (i >= cnt)
        return;
    Chunk<S::V, S::NT> cur[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int idx = i + u * G;
        if (idx < cnt)
            cur[u].load(base + (kbase + list[idx]) * N);
        else
            cur[u].zero();
    }
    for (i += U * G; i < cnt; i += U * G) {
        Chunk<S::V, S::NT> nxt[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int idx = i + u * G;
            if (idx < cnt)
                nxt[u].load(base + (kbase + list[idx]) * N);
            else
                nxt[u].zero();
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            cur[u].add(acc);
#pragma unroll
        for (int u = 0; u < U; ++u)
            cur[u] = nxt[u];
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
        cur[u].add(acc);
}

// gather_columns on a buffer resource over the slice's columns (offset 0 =
// column kbase), as a ring of U load slots per lane.  Round r of group g
// takes the U consecutive list positions r * U * G + g * U + [0, U), read
// from LDS as U/2 32-bit words.  The lane groups of a wave run the same
// number of rounds (that of the wave's first group, which has the most
// positions); positions past the list load zeros.  The list must hold U * G
// readable entries past its end (list_lds reserves them).
template <class S>
__device__ inline void gather_ring(__amdgpu_buffer_rsrc_t w, uint32_t N, uint32_t n_lane, bool lane_in_range,
                                   const uint16_t* list, int cnt, int32_t (&acc)[S::V])
{
    constexpr int G = S::kGroups;
    constexpr int U = S::U;
    constexpr int STEP = U * G;
    static_assert(U % 2 == 0, "list entries are read in pairs");
#pragma unroll
    for (int j = 0; j < S::V; ++j)
        acc[j] = 0;
    const int g = threadIdx.x / S::LG;
    const int g_first = __builtin_amdgcn_readfirstlane(g);
    const int rounds = cnt > g_first * U ? (cnt - g_first * U + STEP - 1) / STEP : 0;
    const uint32_t* pairs = reinterpret_cast<const uint32_t*>(list + g * U);
    // byte offsets of round r's columns in this lane's run; positions past
    // the list get an offset past the resource.  (Masks, not selects: a
    // select of a loaded value would be turned into a branch around the load.)
    auto offsets = [&](int r, uint32_t (&off)[U]) {
        uint32_t two[U / 2];
#pragma unroll
        for (int i = 0; i < U / 2; ++i)
            two[i] = pairs[r * (STEP / 2) + i];
        const int p0 = r * STEP + g * U;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t col = u % 2 ? two[u / 2] >> 16 : two[u / 2] & 0xffffu;
            const uint32_t keep = (p0 + u < cnt && lane_in_range) ? ~0u : 0u;
            off[u] = ((__umul24(col, N) + n_lane) & keep) | (kOutOfRange & ~keep);  // col * N < 2^31
        }
    };
    BufChunk<S::V, S::NT> slot[U];
    {
        uint32_t off[U];
        offsets(0, off);
#pragma unroll
        for (int u = 0; u < U; ++u)
            slot[u].load(w, off[u]);
    }
    // The scheduling barriers keep every slot's refill after its add, so a
    // slot's old and new values never live at once (no register copies) and
    // U loads stay in flight; the round's list entries are read first.
    if constexpr (S::I16) {
        // 16-bit partials, folded into acc every kI16MaxAdds columns (the
        // count is per wave: every lane adds U columns, real or zero, per round)
        uint32_t p16[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        int n16 = 0;
        for (int r = 1; r < rounds; ++r) {
            uint32_t off[U];
            offsets(r, off);
            if (n16 == kI16MaxAdds) {
                flush_i16(acc, p16, n16);
                n16 = 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                slot[u].add_i16(p16);
                slot[u].load(w, off[u]);
                __builtin_amdgcn_sched_barrier(0);
            }
            n16 += U;
        }
        if (rounds > 0) {
            if (n16 == kI16MaxAdds) {
                flush_i16(acc, p16, n16);
                n16 = 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                slot[u].add_i16(p16);
            n16 += U;
        }
        flush_i16(acc, p16, n16);
    } else {
        for (int r = 1; r < rounds; ++r) {
            uint32_t off[U];
            offsets(r, off);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                slot[u].add(acc);
                slot[u].load(w, off[u]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (rounds > 0) {
#pragma unroll
            for (int u = 0; u < U; ++u)
                slot[u].add(acc);
        }
    }
}

// Output of one unit: either FP32 y (ACC == false) or the raw INT32 sums.
template <bool ACC>
__device__ inline void store_result(float* out_row, int32_t* acc_row, const float* __restrict__ scale, int64_t n,
                                    int32_t sum)
{
    if constexpr (ACC) {
        acc_row[n] = sum;
    } else {
        const float as_float = (float)sum;  // exact for |sum| < 2^24, RNE beyond
        out_row[n] = as_float * scale[n];   // one binary32 multiply
    }
}

// The outputs of one tile: the waves' partial sums (red[q * TB + e] for
// wave q and channel n_tile0 + e) are added and written, as FP32 y or raw
// INT32 sums.  Where N, the output row and the scales allow it, each thread
// handles four channels with 16-byte LDS reads, scale loads and nontemporal
// stores: a tile then costs two store instructions instead of eight, and
// narrow stores stall the in-order vector memory pipeline of the CU (every
// weight load queued behind a store waits with it).

template <class S, bool ACC>
__device__ inline void finish_tile(const int32_t* red, int64_t n_tile0, int N, const float* __restrict__ scale,
                                   float* out_row, int32_t* acc_row)
{
    constexpr int TB = S::kTile;
    constexpr int kWaves = S::BLOCK / 64;
    const uintptr_t dst = ACC ? reinterpret_cast<uintptr_t>(acc_row) : reinterpret_cast<uintptr_t>(out_row);
    const uintptr_t sc = ACC ? 0 : reinterpret_cast<uintptr_t>(scale);
    if (TB % 4 == 0 && N % 4 == 0 && ((dst | sc) & 15) == 0) {
        for (int e = 4 * (int)threadIdx.x; e < TB && n_tile0 + e < N; e += 4 * S::BLOCK) {
            i32x4 sum = *reinterpret_cast<const i32x4*>(red + e);
#pragma unroll
            for (int q = 1; q < kWaves; ++q)
                sum += *reinterpret_cast<const i32x4*>(red + q * TB + e);
            if constexpr (ACC) {
                __builtin_nontemporal_store(sum, reinterpret_cast<i32x4*>(acc_row + n_tile0 + e));
            } else {
                const f32x4 s4 = *reinterpret_cast<const f32x4*>(scale + n_tile0 + e);
                f32x4 y;
                y.x = (float)sum.x * s4.x;  // per channel: one exact-or-RNE conversion, one binary32 multiply
                y.y = (float)sum.y * s4.y;
                y.z = (float)sum.z * s4.z;
                y.w = (float)sum.w * s4.w;
                __builtin_nontemporal_store(y, reinterpret_cast<f32x4*>(out_row + n_tile0 + e));
            }
        }
        return;
    }
    for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += S::BLOCK) {
        int32_t sum = 0;
#pragma unroll
        for (int q = 0; q < kWaves; ++q)
            sum += red[q * TB + e];
        store_result<ACC>(out_row, acc_row, scale, n_tile0 + e, sum);
    }
}

// Dynamic LDS of a unit: the active list (uint16 per bit of the slice) and
// the partial sums of every wave.  With one tile per unit the two share the
// same bytes (the list is dead before the reduction).
template <class S>
constexpr size_t list_lds(int slice_words)
{
    // every bit of the slice, plus one round of the ring gather past the end
    return (((size_t)slice_words * 64 + S::U * S::kGroups) * sizeof(uint16_t) + 15) / 16 * 16;
}
template <class S>
constexpr size_t red_lds()
{
    return (size_t)(S::BLOCK / 64) * S::kTile * sizeof(int32_t);
}
template <class S>
constexpr size_t unit_dyn_lds(int slice_words, int tiles_per_unit)
{
    const size_t l = list_lds<S>(slice_words), r = red_lds<S>();
    return tiles_per_unit == 1 ? (l > r ? l : r) : l + r;
}

// Weight and scale pointers of one (weight set, projection) of a
// multi-projection stream: the stream's device operand table holds one per
// handle, set-major.
struct StreamOperands {
    const int8_t* W;
    const float* scale;
};

// Per-projection layout of a token, passed by value as a kernel argument so
// that a workgroup can start loading its spike words before the descriptor
// (weight and scale pointers) has arrived from memory.
constexpr int kStreamMaxProj = 64;
struct StreamLayout {
    int32_t K[kStreamMaxProj];
    int32_t mask_off[kStreamMaxProj];  // word offset of the projection's row within a token
};

// Many independent batch-1 projections in one launch: unit id -> (token,
// projection, tile group); each unit walks the whole K axis of its row, so
// no cross-unit reduction is needed.
// Weight and scale pointers of a unit, given directly or read from a
// stream descriptor once the spike words have been requested.
struct DirectOperands {
    const int8_t* W;
    const float* scale;
    __device__ const int8_t* weights() const { return W; }
    __device__ const float* scales() const { return scale; }
};
__device__ inline DirectOperands operands_of(const DirectOperands& d) { return d; }
__device__ inline DirectOperands operands_of(const StreamOperands* d) { return DirectOperands{d->W, d->scale}; }

// One unit: K-slice [w0, w0 + nw) of one row, tiles [tile0, tile0 + n_tiles_here).
// BUF: weight loads through a buffer resource (needs K * N <= kBufMaxBytes).
template <class S, bool ACC, bool BUF, class Src>
__device__ inline void run_unit(const Src& src, int K, int N, const uint64_t* __restrict__ row, int w0, int nw,
                                int tile0, int n_tiles_here, int n_slices, int32_t* ws_row, uint32_t* counters_row,
                                float* out_row, int32_t* acc_row, SliceLds<S::BLOCK>& s, uint8_t* dyn)
{
    constexpr int TB = S::kTile;
    constexpr int kWaves = S::BLOCK / 64;
    uint16_t* list = reinterpret_cast<uint16_t*>(dyn);
    ThreadWords<S::BLOCK> tw;
    load_words<S::BLOCK>(row, w0, nw, K, tw);
    const DirectOperands ops = operands_of(src);
    const int8_t* __restrict__ W = ops.weights();
    const float* __restrict__ scale = ops.scales();
    const int cnt = compact_words<S::BLOCK>(tw, nw, s, [&](int pos, int k) { list[pos] = (uint16_t)k; });
    int32_t* red = reinterpret_cast<int32_t*>(n_tiles_here == 1 ? dyn : dyn + list_lds<S>(nw));

    const int lg = threadIdx.x % S::LG;
    const int lane = threadIdx.x % 64;
    const int wave = threadIdx.x / 64;
    // the slice's columns [64 w0, K) as a buffer resource (unused without BUF)
    const __amdgpu_buffer_rsrc_t wres = weight_resource(W + 64ll * w0 * N, BUF ? (int64_t)(K - 64 * w0) * N : 0);
    for (int tt = 0; tt < n_tiles_here; ++tt) {
        const int tile = tile0 + tt;
        const int64_t n_tile0 = (int64_t)tile * TB;
        const int64_t n_lane = n_tile0 + (int64_t)lg * S::V;
        int32_t acc[S::V];
        if constexpr (BUF)
            gather_ring<S>(wres, (uint32_t)N, (uint32_t)n_lane, n_lane < N, list, cnt, acc);
        else
            gather_columns<S>(W, N, 64ll * w0, n_lane, n_lane < N, list, cnt, acc);
        // the lane groups of a wave are folded into its first group
#pragma unroll
        for (int d = S::LG; d < 64; d <<= 1)
#pragma unroll
            for (int j = 0; j < S::V; ++j)
                acc[j] += __shfl_xor(acc[j], d, 64);
        __syncthreads();  // list dead (one tile) / previous tile's reduction read
        if (lane < S::LG) {
#pragma unroll
            for (int j = 0; j < S::V; ++j)
                red[wave * TB + lg * S::V + j] = acc[j];
        }
        __syncthreads();

        if (n_slices == 1) {
            finish_tile<S, ACC>(red, n_tile0, N, scale, out_row, acc_row);
            continue;
        }

        // Several K-slices share this tile: exact INT32 atomics into the workspace.
        if (cnt > 0) {
            for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += S::BLOCK) {
                int32_t sum = 0;
#pragma unroll
                for (int q = 0; q < kWaves; ++q)
                    sum += red[q * TB + e];
                atomicAdd(ws_row + n_tile0 + e, sum);
            }
        }
        wait_writes_done();  // this unit's atomic adds are performed before it is counted
        __syncthreads();
        if (threadIdx.x == 0)
            s.is_last = atomicAdd(counters_row + tile, 1u) == (uint32_t)(n_slices - 1);
        __syncthreads();
        if (s.is_last) {
            for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += S::BLOCK) {
                const int32_t sum = atomicExch(ws_row + n_tile0 + e, 0);  // read and re-zero
                store_result<ACC>(out_row, acc_row, scale, n_tile0 + e, sum);
            }
            if (threadIdx.x == 0)
                atomicExch(counters_row + tile, 0u);
        }
    }
}

// One launch of B spike rows against one weight matrix: unit id ->
// (row b, tile group, slice), slices fastest.  A unit covers tiles_per_unit
// consecutive tiles (the last group may hold fewer).
template <class S, bool ACC, bool BUF>
__global__ __launch_bounds__(S::BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void k_gather(const int8_t* __restrict__ W, const float* __restrict__ scale,
                                                     int K, int N, const uint64_t* __restrict__ mask, int wpr,
                                                     int slice_words, int n_slices, int n_tiles, int tiles_per_unit,
                                                     int32_t* ws, uint32_t* counters, int counter_stride,
                                                     float* out, int32_t* acc_out)
{
    __shared__ SliceLds<S::BLOCK> s;
    extern __shared__ __align__(16) uint8_t dyn[];
    const int n_groups = (n_tiles + tiles_per_unit - 1) / tiles_per_unit;
    const int unit = blockIdx.x;
    const int slice = unit % n_slices;
    const int rest = unit / n_slices;
    const int tg = rest % n_groups;
    const int b = rest / n_groups;
    const int w0 = slice * slice_words;
    const int nw = min(slice_words, wpr - w0);
    const int tile0 = tg * tiles_per_unit;
    const int nt = min(tiles_per_unit, n_tiles - tile0);
    const int64_t rowN = (int64_t)b * N;
    run_unit<S, ACC, BUF>(DirectOperands{W, scale}, K, N, mask + (int64_t)b * wpr, w0, nw, tile0, nt, n_slices,
                     n_slices > 1 ? ws + rowN : nullptr,
                     n_slices > 1 ? counters + (int64_t)b * counter_stride : nullptr, ACC ? nullptr : out + rowN,
                     ACC ? acc_out + rowN : nullptr, s, dyn);
}

template <class S, bool BUF>
__global__ __launch_bounds__(S::BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void k_stream(
    const StreamOperands* __restrict__ desc, const StreamLayout layout, int n_proj, int n_sets, int N, int n_tiles,
    int tiles_per_unit, int n_items, int xcd_spread, const uint64_t* __restrict__ masks, int64_t mask_stride,
    float* out, int64_t out_stride)
{
    __shared__ SliceLds<S::BLOCK> s;
    extern __shared__ __align__(16) uint8_t dyn[];
    const int n_groups = (n_tiles + tiles_per_unit - 1) / tiles_per_unit;
    const int n_units = n_items * n_groups;
    int unit = blockIdx.x;
    if (xcd_spread > 1) {
        // Workgroups are dispatched to the XCDs round-robin (block b to XCD
        // b % xcd_spread, in order).  XCD x runs the contiguous unit range
        // [x * per, (x + 1) * per): every XCD then gets the same mix of
        // projections (TCAM and down items differ 4x in work; plain order
        // gives some XCDs twice the down tiles of others), and the tiles of
        // one item run back to back on one XCD, whose L2 keeps their spike
        // words.
        const int per = (n_units + xcd_spread - 1) / xcd_spread;
        unit = (blockIdx.x % xcd_spread) * per + blockIdx.x / xcd_spread;
        if (unit >= n_units)
            return;
    }
    const int tg = unit % n_groups;
    const int item = unit / n_groups;
    const int t = item / n_proj;
    const int j = item - t * n_proj;
    const int K = layout.K[j];
    const uint64_t* row = masks + (int64_t)t * mask_stride + layout.mask_off[j];
    const StreamOperands* d = desc + (t % n_sets) * n_proj + j;  // read after the spike words are requested
    const int tile0 = tg * tiles_per_unit;
    const int nt = min(tiles_per_unit, n_tiles - tile0);
    run_unit<S, false, BUF>(d, K, N, row, 0, (K + 63) / 64, tile0, nt, 1, nullptr, nullptr,
                       out + (int64_t)t * out_stride + (int64_t)j * N, nullptr, s, dyn);
}

// Standalone active-index extraction: one workgroup per row, chunks of
// kMaxSliceWords words, indices written ascending to idx[b*K + i].
constexpr int kCompactBlock = 256;
__global__ __launch_bounds__(kCompactBlock) void k_compact(const uint64_t* __restrict__ mask, int K, int wpr,
                                                           int32_t* __restrict__ idx, int32_t* __restrict__ count)
{
    __shared__ SliceLds<kCompactBlock> s;
    const int b = blockIdx.x;
    const uint64_t* row = mask + (int64_t)b * wpr;
    int32_t* out = idx + (int64_t)b * K;
    int base = 0;
    for (int w0 = 0; w0 < wpr; w0 += kMaxSliceWords) {
        const int nw = min(kMaxSliceWords, wpr - w0);
        const int kb = 64 * w0;
        const int off = base;
        base += compact_slice<kCompactBlock>(row, w0, nw, K, s, [&](int pos, int k) { out[off + pos] = kb + k; });
    }
    if (threadIdx.x == 0)
        count[b] = base;
}

}  // namespace spk
