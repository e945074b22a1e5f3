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
//      column indices in LDS (popcount + wavefront prefix scan, then each
//      wave scatters the set bits of one word with mbcnt);
//   2. gather: lane groups walk the list; every lane streams V bytes of each
//      active column (one coalesced global load per column) and adds the
//      sign-extended bytes into V INT32 registers (one VALU op per byte).
//      Loads are software-pipelined: the next U columns are in flight while
//      the current U are added;
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

constexpr int kMaxSliceWords = 256;  // mask words per K-slice (16384 columns)

template <int BLOCK>
struct SliceLds {
    static_assert(BLOCK % 64 == 0 && BLOCK >= 64 && BLOCK <= 1024, "block must be whole waves");
    static constexpr int kWaves = BLOCK / 64;
    uint64_t words[kMaxSliceWords];
    int32_t offset[kMaxSliceWords];
    int32_t wave_total[kWaves];
    int32_t is_last;
};

// Active positions of mask words [w0, w0 + nw) of one row, ascending.  Bits at
// or above K are dropped.  emit(pos, k_rel) is called once per active bit with
// its rank pos in the list and its index k_rel relative to bit 64*w0.
// Returns |A| of the slice in every thread.  Requires nw <= kMaxSliceWords.
template <int BLOCK, class Emit>
__device__ inline int compact_slice(const uint64_t* __restrict__ row, int w0, int nw, int K, SliceLds<BLOCK>& s,
                                    Emit emit)
{
    constexpr int kWaves = SliceLds<BLOCK>::kWaves;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    // each thread owns a contiguous run of words (one word when BLOCK >= nw),
    // so the scan over threads is a scan in word order
    const int per = (nw + BLOCK - 1) / BLOCK;
    const int first = t * per;
    const int last = min(first + per, nw);
    int pc = 0;
    for (int i = first; i < last; ++i) {
        const int w = w0 + i;
        uint64_t word = row[w];
        const int valid = K - 64 * w;  // bits of this word below K
        if (valid < 64)
            word &= valid <= 0 ? 0ull : ((1ull << valid) - 1ull);
        s.words[i] = word;
        pc += __popcll(word);
    }
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
    int off = before + incl - pc;  // exclusive prefix of this thread's words
    for (int i = first; i < last; ++i) {
        s.offset[i] = off;
        off += __popcll(s.words[i]);
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
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

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

__device__ inline void add_i8x4(int32_t* acc, uint32_t d)
{
    acc[0] += (int32_t)(int8_t)(d & 0xffu);
    acc[1] += (int32_t)(int8_t)((d >> 8) & 0xffu);
    acc[2] += (int32_t)(int8_t)((d >> 16) & 0xffu);
    acc[3] += ((int32_t)d) >> 24;
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

// Launch shape.  Lane groups of LG lanes (a group may span waves); a lane
// covers V consecutive output channels, a group one tile of TB = LG * V
// channels of one column at a time; U columns per group are in flight;
// BLOCK threads per workgroup; NT marks weight loads nontemporal.
template <int V_, int LG_, int U_, int BLOCK_, bool NT_ = false>
struct Shape {
    static constexpr int V = V_, LG = LG_, U = U_, BLOCK = BLOCK_;
    static constexpr bool NT = NT_;
    static constexpr int kTile = V * LG;
    static constexpr int kGroups = BLOCK / LG;
    static_assert(BLOCK % LG == 0 && LG >= 1 && LG <= BLOCK, "lane groups must tile the workgroup");
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

// Dynamic LDS of a unit: the active list (uint16 per bit of the slice) and
// the partial sums of every lane group.  With one tile per unit the two
// share the same bytes (the list is dead before the reduction).
template <class S>
constexpr size_t list_lds(int slice_words)
{
    return ((size_t)slice_words * 64 * sizeof(uint16_t) + 15) / 16 * 16;
}
template <class S>
constexpr size_t red_lds()
{
    return (size_t)S::BLOCK * S::V * sizeof(int32_t);
}
template <class S>
constexpr size_t unit_dyn_lds(int slice_words, int tiles_per_unit)
{
    const size_t l = list_lds<S>(slice_words), r = red_lds<S>();
    return tiles_per_unit == 1 ? (l > r ? l : r) : l + r;
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
__device__ inline DirectOperands operands_of(const StreamDesc* d) { return DirectOperands{d->W, d->scale}; }

// One unit: K-slice [w0, w0 + nw) of one row, tiles [tile0, tile0 + n_tiles_here).
template <class S, bool ACC, class Src>
__device__ inline void run_unit(const Src& src, int K, int N, const uint64_t* __restrict__ row, int w0, int nw,
                                int tile0, int n_tiles_here, int n_slices, int32_t* ws_row, uint32_t* counters_row,
                                float* out_row, int32_t* acc_row, SliceLds<S::BLOCK>& s, uint8_t* dyn)
{
    constexpr int TB = S::kTile;
    constexpr int G = S::kGroups;
    uint16_t* list = reinterpret_cast<uint16_t*>(dyn);
    const int cnt = compact_slice<S::BLOCK>(row, w0, nw, K, s, [&](int pos, int k) { list[pos] = (uint16_t)k; });
    const DirectOperands ops = operands_of(src);
    const int8_t* __restrict__ W = ops.weights();
    const float* __restrict__ scale = ops.scales();
    int32_t* red = reinterpret_cast<int32_t*>(n_tiles_here == 1 ? dyn : dyn + list_lds<S>(nw));

    const int lg = threadIdx.x % S::LG;
    const int g = threadIdx.x / S::LG;
    for (int tt = 0; tt < n_tiles_here; ++tt) {
        const int tile = tile0 + tt;
        const int64_t n_tile0 = (int64_t)tile * TB;
        const int64_t n_lane = n_tile0 + (int64_t)lg * S::V;
        int32_t acc[S::V];
        gather_columns<S>(W, N, 64ll * w0, n_lane, n_lane < N, list, cnt, acc);
        __syncthreads();  // list dead (one tile) / previous tile's reduction read
#pragma unroll
        for (int j = 0; j < S::V; ++j)
            red[g * TB + lg * S::V + j] = acc[j];
        __syncthreads();

        if (n_slices == 1) {
            for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += S::BLOCK) {
                int32_t sum = 0;
#pragma unroll
                for (int q = 0; q < G; ++q)
                    sum += red[q * TB + e];
                store_result<ACC>(out_row, acc_row, scale, n_tile0 + e, sum);
            }
            continue;
        }

        // Several K-slices share this tile: exact INT32 atomics into the workspace.
        if (cnt > 0) {
            for (int e = threadIdx.x; e < TB && n_tile0 + e < N; e += S::BLOCK) {
                int32_t sum = 0;
#pragma unroll
                for (int q = 0; q < G; ++q)
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
template <class S, bool ACC>
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
    run_unit<S, ACC>(DirectOperands{W, scale}, K, N, mask + (int64_t)b * wpr, w0, nw, tile0, nt, n_slices,
                     n_slices > 1 ? ws + rowN : nullptr,
                     n_slices > 1 ? counters + (int64_t)b * counter_stride : nullptr, ACC ? nullptr : out + rowN,
                     ACC ? acc_out + rowN : nullptr, s, dyn);
}

template <class S>
__global__ __launch_bounds__(S::BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void k_stream(
    const StreamDesc* __restrict__ desc, const StreamLayout layout, int n_proj, int n_sets, int N, int n_tiles,
    int tiles_per_unit, int n_items, int xcd_spread, const uint64_t* __restrict__ masks, int64_t mask_stride,
    float* out, int64_t out_stride)
{
    __shared__ SliceLds<S::BLOCK> s;
    extern __shared__ __align__(16) uint8_t dyn[];
    const int n_groups = (n_tiles + tiles_per_unit - 1) / tiles_per_unit;
    int tg, item;
    if (xcd_spread > 1) {
        // Workgroups are dispatched round-robin over the XCDs; keep the tile
        // groups of one (token, projection) item on the same XCD.
        const int per = xcd_spread * n_groups;
        const int p = blockIdx.x % per;
        item = (blockIdx.x / per) * xcd_spread + p % xcd_spread;
        tg = p / xcd_spread;
        if (item >= n_items)
            return;
    } else {
        tg = blockIdx.x % n_groups;
        item = blockIdx.x / n_groups;
    }
    const int t = item / n_proj;
    const int j = item - t * n_proj;
    const int K = layout.K[j];
    const uint64_t* row = masks + (int64_t)t * mask_stride + layout.mask_off[j];
    const StreamDesc* d = desc + (t % n_sets) * n_proj + j;  // read after the spike words are requested
    const int tile0 = tg * tiles_per_unit;
    const int nt = min(tiles_per_unit, n_tiles - tile0);
    run_unit<S, false>(d, K, N, row, 0, (K + 63) / 64, tile0, nt, 1, nullptr, nullptr,
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
