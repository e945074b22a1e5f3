// Active-column gather for the spike-gated INT8 projection on CDNA4 (gfx950).
//
// Computes Eq. (sparse) of the paper (Sec. 2.3): for a binary spike row x,
// y[n] = scale[n] * sum_{k in A} Q[n][k] with A = {k : x_k = 1} (Sec. 2.2).
// Weights are column-major (W[k*N + n]), so each active column is one
// contiguous run of N bytes; inactive columns are never read.
//
// One workgroup ("unit") owns a tile of output channels and a slice of the
// K axis for one spike row:
//   1. compaction: the slice's mask words become an ascending list of active
//      column indices in LDS (popcount + wavefront prefix scan, then each
//      wave scatters the set bits of one word with mbcnt);
//   2. gather: lane groups walk the list; every lane streams V bytes of each
//      active column (one coalesced global load per column) and adds the
//      sign-extended bytes into V INT32 registers (one VALU op per byte);
//   3. the lane groups' partial sums are added in LDS;
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

namespace spk {

constexpr int kBlock = 256;                  // threads per workgroup (4 waves)
constexpr int kWaves = kBlock / 64;
constexpr int kMaxSliceWords = kBlock;       // one mask word per thread in the scan
constexpr int kUnroll = 4;                   // columns in flight per lane group

struct SliceLds {
    uint64_t words[kMaxSliceWords];
    int32_t offset[kMaxSliceWords];
    int32_t wave_total[kWaves];
    int32_t is_last;
};

// Active positions of mask words [w0, w0 + nw) of one row, ascending.  Bits at
// or above K are dropped.  emit(pos, k_rel) is called once per active bit with
// its rank pos in the list and its index k_rel relative to bit 64*w0.
// Returns |A| of the slice in every thread.  Requires nw <= kBlock.
template <class Emit>
__device__ inline int compact_slice(const uint64_t* __restrict__ row, int w0, int nw, int K, SliceLds& s,
                                    Emit emit)
{
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    uint64_t word = 0;
    if (t < nw) {
        const int w = w0 + t;
        word = row[w];
        const int valid = K - 64 * w;  // bits of this word below K
        if (valid < 64)
            word &= valid <= 0 ? 0ull : ((1ull << valid) - 1ull);
    }
    const int pc = __popcll(word);
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
    if (t < nw) {
        s.words[t] = word;
        s.offset[t] = before + incl - pc;
    }
    __syncthreads();
    for (int w = wave; w < nw; w += kWaves) {
        const uint64_t wd = s.words[w];
        if (wd == 0)
            continue;
        const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(wd >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)wd, 0));
        if ((wd >> lane) & 1ull)
            emit(s.offset[w] + below, 64 * w + lane);
    }
    __syncthreads();
    return total;
}

// V bytes of one column for one lane, added into V INT32 accumulators.
template <int V>
struct Chunk;

__device__ inline void add_i8x4(int32_t* acc, uint32_t d)
{
    acc[0] += (int32_t)(int8_t)(d & 0xffu);
    acc[1] += (int32_t)(int8_t)((d >> 8) & 0xffu);
    acc[2] += (int32_t)(int8_t)((d >> 16) & 0xffu);
    acc[3] += ((int32_t)d) >> 24;
}

template <>
struct Chunk<16> {
    uint4 v;
    __device__ void load(const int8_t* p) { v = *reinterpret_cast<const uint4*>(p); }
    __device__ void add(int32_t* acc) const
    {
        add_i8x4(acc + 0, v.x);
        add_i8x4(acc + 4, v.y);
        add_i8x4(acc + 8, v.z);
        add_i8x4(acc + 12, v.w);
    }
};
template <>
struct Chunk<8> {
    uint2 v;
    __device__ void load(const int8_t* p) { v = *reinterpret_cast<const uint2*>(p); }
    __device__ void add(int32_t* acc) const
    {
        add_i8x4(acc + 0, v.x);
        add_i8x4(acc + 4, v.y);
    }
};
template <>
struct Chunk<4> {
    uint32_t v;
    __device__ void load(const int8_t* p) { v = *reinterpret_cast<const uint32_t*>(p); }
    __device__ void add(int32_t* acc) const { add_i8x4(acc, v); }
};
template <>
struct Chunk<1> {  // any N, any alignment
    int8_t v;
    __device__ void load(const int8_t* p) { v = *p; }
    __device__ void add(int32_t* acc) const { acc[0] += (int32_t)v; }
};

// Lane groups of LG lanes; a lane covers V consecutive output channels, a
// group covers one tile of TB = LG * V channels of one column at a time.
template <int V, int LG>
struct Geometry {
    static constexpr int kTile = V * LG;
    static constexpr int kGroups = kBlock / LG;
    static_assert(kBlock % LG == 0 && LG <= 64 && (64 % LG) == 0, "lane groups must tile a wave");
};

// Sum the active columns listed in `list` (indices relative to kbase) over
// this lane's V channels starting at byte n_lane of each column.
template <int V, int LG>
__device__ inline void gather_columns(const int8_t* __restrict__ W, int64_t N, int64_t kbase, int64_t n_lane,
                                      bool lane_in_range, const uint16_t* list, int cnt, int32_t (&acc)[V])
{
    constexpr int G = Geometry<V, LG>::kGroups;
#pragma unroll
    for (int j = 0; j < V; ++j)
        acc[j] = 0;
    if (!lane_in_range)
        return;
    const int8_t* base = W + n_lane;
    int i = threadIdx.x / LG;
    for (; i + (kUnroll - 1) * G < cnt; i += kUnroll * G) {
        Chunk<V> c[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            c[u].load(base + (kbase + list[i + u * G]) * N);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            c[u].add(acc);
    }
    for (; i < cnt; i += G) {
        Chunk<V> c;
        c.load(base + (kbase + list[i]) * N);
        c.add(acc);
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

// Bytes of dynamic LDS a unit needs: the active list (uint16 per bit of the
// slice) and, reusing the same space afterwards, the partial sums of every
// lane group.
template <int V, int LG>
constexpr size_t unit_dyn_lds(int slice_words)
{
    const size_t list = (size_t)slice_words * 64 * sizeof(uint16_t);
    const size_t red = (size_t)kBlock * V * sizeof(int32_t);
    return list > red ? list : red;
}

template <int V, int LG, bool ACC>
__device__ inline void run_unit(const int8_t* __restrict__ W, const float* __restrict__ scale, int K, int N,
                                const uint64_t* __restrict__ row, int w0, int nw, int tile, int n_slices,
                                int32_t* ws_row, uint32_t* counter, float* out_row, int32_t* acc_row, SliceLds& s,
                                uint8_t* dyn)
{
    using Geo = Geometry<V, LG>;
    constexpr int TB = Geo::kTile;
    constexpr int G = Geo::kGroups;
    uint16_t* list = reinterpret_cast<uint16_t*>(dyn);
    const int cnt = compact_slice(row, w0, nw, K, s, [&](int pos, int k) { list[pos] = (uint16_t)k; });

    const int lg = threadIdx.x % LG;
    const int g = threadIdx.x / LG;
    const int64_t n_lane = (int64_t)tile * TB + (int64_t)lg * V;
    int32_t acc[V];
    gather_columns<V, LG>(W, N, 64ll * w0, n_lane, n_lane < N, list, cnt, acc);
    __syncthreads();  // the list is dead; reuse its LDS for the reduction

    int32_t* red = reinterpret_cast<int32_t*>(dyn);
#pragma unroll
    for (int j = 0; j < V; ++j)
        red[g * TB + lg * V + j] = acc[j];
    __syncthreads();

    const int64_t n_tile0 = (int64_t)tile * TB;
    if (n_slices == 1) {
        for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += kBlock) {
            int32_t sum = 0;
#pragma unroll
            for (int q = 0; q < G; ++q)
                sum += red[q * TB + e];
            store_result<ACC>(out_row, acc_row, scale, n_tile0 + e, sum);
        }
        return;
    }

    // Several K-slices share this tile: exact INT32 atomics into the workspace.
    if (cnt > 0) {
        for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += kBlock) {
            int32_t sum = 0;
#pragma unroll
            for (int q = 0; q < G; ++q)
                sum += red[q * TB + e];
            atomicAdd(ws_row + n_tile0 + e, sum);
        }
    }
    __threadfence();  // release: this unit's adds are visible before it is counted
    __syncthreads();
    if (threadIdx.x == 0)
        s.is_last = atomicAdd(counter, 1u) == (uint32_t)(n_slices - 1);
    __syncthreads();
    if (!s.is_last)
        return;
    __threadfence();  // acquire: every other slice's adds are visible
    for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += kBlock) {
        const int32_t sum = atomicExch(ws_row + n_tile0 + e, 0);  // read and re-zero
        store_result<ACC>(out_row, acc_row, scale, n_tile0 + e, sum);
    }
    if (threadIdx.x == 0)
        atomicExch(counter, 0u);
}

// One launch of B spike rows against one weight matrix: unit id ->
// (row b, tile, slice), slices fastest.
template <int V, int LG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_gather(const int8_t* __restrict__ W, const float* __restrict__ scale,
                                                   int K, int N, const uint64_t* __restrict__ mask, int wpr,
                                                   int slice_words, int n_slices, int n_tiles, int32_t* ws,
                                                   uint32_t* counters, int counter_stride, float* out,
                                                   int32_t* acc_out)
{
    __shared__ SliceLds s;
    extern __shared__ __align__(16) uint8_t dyn[];
    const int unit = blockIdx.x;
    const int slice = unit % n_slices;
    const int rest = unit / n_slices;
    const int tile = rest % n_tiles;
    const int b = rest / n_tiles;
    const int w0 = slice * slice_words;
    const int nw = min(slice_words, wpr - w0);
    const int64_t rowN = (int64_t)b * N;
    run_unit<V, LG, ACC>(W, scale, K, N, mask + (int64_t)b * wpr, w0, nw, tile, n_slices,
                         n_slices > 1 ? ws + rowN : nullptr,
                         n_slices > 1 ? counters + (int64_t)b * counter_stride + tile : nullptr,
                         ACC ? nullptr : out + rowN, ACC ? acc_out + rowN : nullptr, s, dyn);
}

// Descriptor of one projection in a multi-projection stream.
struct StreamDesc {
    const int8_t* W;
    const float* scale;
    int32_t K;
    int32_t wpr;
    int64_t mask_off;  // word offset of this projection's row within a token
    int64_t out_off;   // float offset of this projection's output within a token
};

// Many independent batch-1 projections in one launch: unit id -> (token,
// projection, tile); each unit walks the whole K axis of its row, so no
// cross-unit reduction is needed.
template <int V, int LG>
__global__ __launch_bounds__(kBlock) void k_stream(const StreamDesc* __restrict__ desc, int n_proj, int n_sets,
                                                   int N, int n_tiles, const uint64_t* __restrict__ masks,
                                                   int64_t mask_stride, float* out, int64_t out_stride)
{
    __shared__ SliceLds s;
    extern __shared__ __align__(16) uint8_t dyn[];
    const int tile = blockIdx.x % n_tiles;
    const int item = blockIdx.x / n_tiles;
    const int t = item / n_proj;
    const int j = item - t * n_proj;
    const StreamDesc d = desc[(t % n_sets) * n_proj + j];
    run_unit<V, LG, false>(d.W, d.scale, d.K, N, masks + (int64_t)t * mask_stride + d.mask_off, 0, d.wpr, tile, 1,
                           nullptr, nullptr, out + (int64_t)t * out_stride + d.out_off, nullptr, s, dyn);
}

// Standalone active-index extraction: one workgroup per row, chunks of
// kBlock words, indices written ascending to idx[b*K + i].
__global__ __launch_bounds__(kBlock) void k_compact(const uint64_t* __restrict__ mask, int K, int wpr,
                                                    int32_t* __restrict__ idx, int32_t* __restrict__ count)
{
    __shared__ SliceLds s;
    const int b = blockIdx.x;
    const uint64_t* row = mask + (int64_t)b * wpr;
    int32_t* out = idx + (int64_t)b * K;
    int base = 0;
    for (int w0 = 0; w0 < wpr; w0 += kBlock) {
        const int nw = min(kBlock, wpr - w0);
        const int kb = 64 * w0;
        const int off = base;
        base += compact_slice(row, w0, nw, K, s, [&](int pos, int k) { out[off + pos] = kb + k; });
    }
    if (threadIdx.x == 0)
        count[b] = base;
}

}  // namespace spk
