// Output-head candidate-row verification (gfx950).
//
// Paper Sec. 5 (projection-only configuration): the vocabulary projection
// runs with INT8 activations over all V rows; when the gap between the two
// largest of those approximate logits is below a threshold, the K
// highest-scoring rows are recomputed with the FP32 activations and the
// token is the best recomputed row; otherwise it is the approximate top row.
//
// k_head_approx: the activation vector is quantized with the Sec. 2.3
// formulas (one scale for the vector, binary32, ties to even), each row's
// integer dot product with the INT8 weights is exact (v_dot4 on four byte
// pairs at a time, INT32), and the logit is fl32(fl32(acc) * fl32(s_m * s_x)).
// The work split is the dense register kernel's: 32 lanes per row, each
// lane's activation slice held in registers (here as packed INT8), a ring of
// U rows of 16-byte weight loads in flight, rows q + Gq r per lane group,
// results parked in lanes and stored 32 rows at a time.
//
// At the end of k_head_approx each workgroup lists its four largest logits
// and the largest key it leaves out.  When the gate can ask for verification
// (threshold > 0), every row's FP32-activation logit is computed in the same
// pass from the same weight registers, in the dense register kernel's order
// (bit for bit that kernel's output for the row), and the listed rows carry
// theirs: the candidates need no second read of their weights.
//
// k_head_select: one workgroup of 1024 threads.  The KK = max(K, 2) largest
// logits are found on order-preserving 32-bit keys: a lower bound L on the
// KK-th largest comes from the workgroup maxima, the listed entries at or
// above L (about a hundred for KK = 64, a few dozen for KK = 16) are pooled
// in LDS and each is placed by its rank among them (equal logits by
// ascending row).  The lists suffice
// when every key they leave out is below the KK-th selected key; otherwise
// the whole array is scanned (pooling, or past 1024 entries a radix select
// with digits of 11, 11 and 10 bits).  It then computes the gap
// fl32(l(1) - l(2)) and, when it is below the threshold, takes the K
// candidates' FP32-activation logits (per lane an FMA chain over its 16-byte
// chunks l + 32 j, the 32-lane tree, one multiply by s_m) from the lists, or
// computes them itself in the same order after a whole-array selection, and
// picks the largest (ties: the lower row).
//
// Reading the 57,344 logits, or the 64 candidate rows, from memory in one
// workgroup is bound by the misses one compute unit keeps in flight; the
// lists cut the first to 28 KB and the fused FP32 logits remove the second
// whenever the lists suffice.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "buffer.hpp"
#include "dense.hpp"  // group32_sum's DPP helpers, kRegLanes, kRegGroups, kRegBlock

namespace spk {

constexpr int kHeadMaxK = 64;          // candidates
constexpr int kSelectBlock = 1024;     // threads of a selecting workgroup
constexpr int kHeadMaxChunks = 16;     // K <= 16 * 256 = 4096 in the recompute
constexpr int kListLen = 4;            // largest logits each approximate-head workgroup lists

template <int CTRL>
__device__ inline int add_dpp_int(int v)
{
    return v + __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}

// Exact INT32 sum over the 32 lanes of a group (every lane gets it).
__device__ inline int group32_sum_int(int v)
{
    v = add_dpp_int<0xB1>(v);
    v = add_dpp_int<0x4E>(v);
    v = add_dpp_int<0x141>(v);
    v = add_dpp_int<0x140>(v);
    return v + __builtin_amdgcn_ds_swizzle(v, 0x401F);
}

__device__ inline int8_t quant_act(float v, float s)
{
    return (int8_t)fminf(fmaxf(__builtin_rintf(__fdiv_rn(v, s)), -127.0f), 127.0f);
}

// s_x of the activation vector and its quantized copy in LDS, computed by the
// whole workgroup: thread t holds elements t + BLOCK i (i < PER, K <= BLOCK
// PER), all loaded at once (zeros past K), so the quantization needs no
// second read of x.
template <int BLOCK, int PER>
__device__ inline float quantize_activations(const float* __restrict__ x, int K, float* red, int8_t* xq_lds)
{
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(x), 0, K * 4, kBufferFlags);
    float xv[PER];
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        xv[i] = __builtin_bit_cast(float,
                                   __builtin_amdgcn_raw_buffer_load_b32(xres, (threadIdx.x + BLOCK * i) * 4, 0, 0));
        amax = fmaxf(amax, fabsf(xv[i]));
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1)
        amax = fmaxf(amax, __shfl_xor(amax, d, 64));
    if (threadIdx.x % 64 == 0)
        red[threadIdx.x / 64] = amax;
    __syncthreads();
    float m = red[0];
#pragma unroll
    for (int w = 1; w < BLOCK / 64; ++w)
        m = fmaxf(m, red[w]);
    const float sx = __fdiv_rn(fmaxf(m, 1e-8f), 127.0f);
#pragma unroll
    for (int i = 0; i < PER; ++i)
        if (threadIdx.x + BLOCK * i < K)
            xq_lds[threadIdx.x + BLOCK * i] = quant_act(xv[i], sx);
    __syncthreads();
    return sx;
}

// Order-preserving key of a float: larger floats give larger keys.
__device__ inline uint32_t order_key(float f)
{
    const uint32_t u = __builtin_bit_cast(uint32_t, f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float key_value(uint32_t k)
{
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __builtin_bit_cast(float, u);
}

template <int CTRL>
__device__ inline uint32_t max_dpp(uint32_t v)
{
    return max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false));
}

// Maximum over the 64 lanes, in every lane: DPP within each row of 16 lanes,
// then the four row results read as scalars.
__device__ inline uint32_t wave_max_u32(uint32_t v)
{
    v = max_dpp<0xB1>(v);   // lane ^ 1
    v = max_dpp<0x4E>(v);   // lane ^ 2
    v = max_dpp<0x141>(v);  // the other quad of 8
    v = max_dpp<0x140>(v);  // the other 8 of 16
    const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return max(max(r0, r1), max(r2, r3));
}

// FP32 logit of one row with the FP32 activations, computed by one wave in
// the dense register kernel's order, so the result is bit for bit that
// kernel's output for the row: lane l of each half-wave covers the 16-byte
// chunks l + 32 j of the row (j < ceil(K / 512)), one FMA chain over its
// chunks (j, then byte order), the 32-lane tree, one multiply by the row's
// scale.  Chunks are loaded four at a time (one batch up to K = 2048).
// Both half-waves compute it; every lane returns the result.
__device__ inline float recompute_row(const int8_t* __restrict__ Q, const float* __restrict__ scale, int K,
                                      const float* __restrict__ x, int row)
{
    constexpr int kBatch = 4;
    const int l = threadIdx.x % kRegLanes;
    const int n_chunks = K / 16;
    const int n_j = (n_chunks + kRegLanes - 1) / kRegLanes;
    const int8_t* qrow = Q + (int64_t)row * K;
    const float s = scale[row];
    float acc = 0.0f;
    for (int j0 = 0; j0 < n_j; j0 += kBatch) {
        u32x4 qd[kBatch];
        f32x4 xv[kBatch][4];
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            const int c = l + kRegLanes * (j0 + b);
            const bool ok = j0 + b < n_j && c < n_chunks;
            qd[b] = ok ? *reinterpret_cast<const u32x4*>(qrow + 16 * c) : u32x4{0, 0, 0, 0};  // Q 16-byte aligned
#pragma unroll
            for (int t = 0; t < 4; ++t)
                xv[b][t] = ok ? f32x4{x[16 * c + 4 * t], x[16 * c + 4 * t + 1], x[16 * c + 4 * t + 2],
                                      x[16 * c + 4 * t + 3]}
                              : f32x4{0.0f, 0.0f, 0.0f, 0.0f};  // x is 4-byte aligned
        }
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            if (j0 + b < n_j && l + kRegLanes * (j0 + b) < n_chunks) {
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t d = qd[b][t];
                    acc = __builtin_fmaf(cvt_i8<0>(d), xv[b][t].x, acc);
                    acc = __builtin_fmaf(cvt_i8<1>(d), xv[b][t].y, acc);
                    acc = __builtin_fmaf(cvt_i8<2>(d), xv[b][t].z, acc);
                    acc = __builtin_fmaf(cvt_i8<3>(d), xv[b][t].w, acc);
                }
            }
        }
    }
    return group32_sum(acc) * s;
}

// Device workspace of one head verification: written by the approximate
// head, read by the selection of the same call (no state across calls).
// Workgroup b of the approximate head owns slot (b % 16) 64 + b / 16 of each
// array, the slot that thread b / 16 of wave b % 16 of the selecting
// workgroup reads, so that the lists spread evenly over its 16 waves and
// each wave's loads are contiguous.
constexpr int kApproxMaxWgs = 512;   // the approximate head's grid is at most this
constexpr int kListSlots = 1024;     // one per selecting thread
__device__ inline int list_slot(int b)
{
    return (b % 16) * 64 + b / 16;
}
struct HeadWorkspace {
    // per approximate-head workgroup: its kListLen largest logits (key << 32 |
    // row, largest first, key 0: none), then the largest key it does not list
    uint64_t lists[kListLen + 1][kListSlots];
    // the listed rows recomputed with the FP32 activations (when the gate can
    // ask for verification)
    float list_rec[kListLen][kListSlots];
};

template <int NPL, int U, bool SPEC>
__global__ __launch_bounds__(kRegBlock) void k_head_approx(const int8_t* __restrict__ Q, const float* __restrict__ scale,
                                                           int K, int V, const float* __restrict__ x,
                                                           float* __restrict__ logits, HeadWorkspace* __restrict__ ws)
{
    __shared__ float red[kRegBlock / 64];
    __shared__ uint64_t wave_best[kRegBlock / 64][kListLen];
    __shared__ uint32_t wave_next[kRegBlock / 64];
    __shared__ __align__(16) int8_t xq_lds[kHeadMaxChunks * 256];  // the quantized activations
    const int l = threadIdx.x % kRegLanes;
    const int q = blockIdx.x * kRegGroups + threadIdx.x / kRegLanes;
    const int Gq = gridDim.x * kRegGroups;
    const int q_wave = q & ~1;
    const int n_steps = __builtin_amdgcn_readfirstlane(q_wave < V ? (V - q_wave + Gq - 1) / Gq : 0);
    const int n_chunks = K / 16;
    const __amdgpu_buffer_rsrc_t qres = weight_resource(Q, (int64_t)V * K);
    const __amdgpu_buffer_rsrc_t sres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(scale), 0, V * 4, kBufferFlags);

    uint32_t chunk_off[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int c = l + kRegLanes * j;
        chunk_off[j] = c < n_chunks ? (uint32_t)(c * 16) : 0u;
    }
    auto row_base = [&](int r) -> uint32_t {
        const int m = q + Gq * r;
        return r < n_steps && m < V ? (uint32_t)m * (uint32_t)K : kOutOfRange;
    };
    // the first ring of weight loads goes out before the activation prologue
    u32x4 slot[U][NPL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t base = row_base(u);
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            slot[u][j] = __builtin_amdgcn_raw_buffer_load_b128(qres, base + chunk_off[j], 0, 2);
    }
    // SPEC: this lane's FP32 activations x[16 c + t] for its chunks c (zeros
    // past K), as the dense register kernel holds them
    float xr[SPEC ? NPL : 1][16];
    if constexpr (SPEC) {
        const __amdgpu_buffer_rsrc_t xres =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(x), 0, K * 4, kBufferFlags);
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int c = l + kRegLanes * j;
            const uint32_t base = c < n_chunks ? (uint32_t)(c * 16) * 4u : kOutOfRange;
#pragma unroll
            for (int t = 0; t < 16; ++t)
                xr[j][t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, base + 4 * t, 0, 0));
        }
    }
    // the vector quantized once per workgroup (K <= 512 NPL), then this
    // lane's activations as packed INT8 (zeros past K)
    const float sx = quantize_activations<kRegBlock, 512 * NPL / kRegBlock>(x, K, red, xq_lds);
    uint32_t xq[NPL][4];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int c = l + kRegLanes * j;
        const u32x4 v = c < n_chunks ? *reinterpret_cast<const u32x4*>(xq_lds + 16 * c) : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 4; ++i)
            xq[j][i] = v[i];
    }
    auto scale_of_step = [&](int rr) -> float {
        const int m = q + Gq * rr;
        const uint32_t off = rr < n_steps && m < V ? (uint32_t)m * 4u : kOutOfRange;
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sres, off, 0, 0));
    };
    float sc = scale_of_step(l);
    int parked = 0;
    float parked32 = 0.0f;  // SPEC: the row's FP32-activation sum
    // this lane's five largest stored logits, largest first (key 0: none),
    // with (SPEC) their rows' FP32-activation logits
    uint32_t tk[kListLen + 1] = {};
    int trow[kListLen + 1] = {};
    float tval[kListLen + 1] = {};
    for (int r0 = 0; r0 < n_steps; r0 += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = r0 + u;
            int acc = 0;
#pragma unroll
            for (int j = 0; j < NPL; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc = __builtin_amdgcn_sdot4((int)slot[u][j][i], (int)xq[j][i], acc, false);
            float acc32 = 0.0f;
            if constexpr (SPEC) {
                // the dense register kernel's chain: chunks j, then byte order
#pragma unroll
                for (int j = 0; j < NPL; ++j)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const uint32_t d = slot[u][j][i];
                        acc32 = __builtin_fmaf(cvt_i8<0>(d), xr[j][4 * i + 0], acc32);
                        acc32 = __builtin_fmaf(cvt_i8<1>(d), xr[j][4 * i + 1], acc32);
                        acc32 = __builtin_fmaf(cvt_i8<2>(d), xr[j][4 * i + 2], acc32);
                        acc32 = __builtin_fmaf(cvt_i8<3>(d), xr[j][4 * i + 3], acc32);
                    }
            }
            {
                const uint32_t base = row_base(r + U);
#pragma unroll
                for (int j = 0; j < NPL; ++j)
                    slot[u][j] = __builtin_amdgcn_raw_buffer_load_b128(qres, base + chunk_off[j], 0, 2);
            }
            __builtin_amdgcn_sched_barrier(0);
            const int tot = group32_sum_int(acc);
            if (l == (r & 31))
                parked = tot;
            if constexpr (SPEC) {
                const float tot32 = group32_sum(acc32);
                if (l == (r & 31))
                    parked32 = tot32;
            }
            if (r < n_steps && ((r & 31) == 31 || r == n_steps - 1)) {
                const int rr = (r & ~31) + l;
                const int m = q + Gq * rr;
                if (rr <= r && m < V) {
                    const float c = sc * sx;
                    const float lg = (float)parked * c;
                    logits[m] = lg;
                    uint32_t ck = order_key(lg);
                    int cr = m;
                    float cv = SPEC ? parked32 * sc : 0.0f;  // the dense kernel's y for row m
#pragma unroll
                    for (int i = 0; i <= kListLen; ++i) {  // insertion, larger keys first
                        const bool up = ck > tk[i];
                        const uint32_t ok = tk[i];
                        const int orow = trow[i];
                        const float oval = tval[i];
                        tk[i] = up ? ck : ok;
                        trow[i] = up ? cr : orow;
                        tval[i] = up ? cv : oval;
                        ck = up ? ok : ck;
                        cr = up ? orow : cr;
                        cv = up ? oval : cv;
                    }
                }
                sc = scale_of_step((r & ~31) + 32 + l);
            }
        }
    }
    // The workgroup's four largest logits and the largest key it leaves out:
    // each wave pops its lanes' heads five times, then wave 0 merges the
    // waves' entries the same way.  The selection takes the candidates from
    // these lists.  With SPEC (a gate that can ask for verification) the
    // listed rows' FP32-activation logits go with them.
    __shared__ float wave_bval[kRegBlock / 64][kListLen];
    const int lane64 = threadIdx.x % 64, wv = threadIdx.x / 64;
    uint64_t best[kListLen];
    float bval[kListLen];
    uint32_t next = 0;
#pragma unroll
    for (int r = 0; r <= kListLen; ++r) {
        const uint32_t m = wave_max_u32(tk[0]);
        const int h = __ffsll((unsigned long long)__ballot(tk[0] == m)) - 1;
        const int hrow = __builtin_amdgcn_readlane(trow[0], h);
        const float hval = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, tval[0]), h));
        if (r < kListLen) {
            best[r] = (uint64_t)m << 32 | (uint32_t)hrow;
            bval[r] = hval;
        } else {
            next = m;
        }
        if (lane64 == h) {
#pragma unroll
            for (int i = 0; i < kListLen; ++i) {
                tk[i] = tk[i + 1];
                trow[i] = trow[i + 1];
                tval[i] = tval[i + 1];
            }
            tk[kListLen] = 0;
        }
    }
    if (lane64 == 0) {
#pragma unroll
        for (int r = 0; r < kListLen; ++r) {
            wave_best[wv][r] = best[r];
            wave_bval[wv][r] = bval[r];
        }
        wave_next[wv] = next;
    }
    __syncthreads();
    const int my_slot = list_slot(blockIdx.x);
    if (wv == 0) {
        const uint64_t e = lane64 < (kRegBlock / 64) * kListLen ? wave_best[lane64 / kListLen][lane64 % kListLen] : 0ull;
        const float ev = lane64 < (kRegBlock / 64) * kListLen ? wave_bval[lane64 / kListLen][lane64 % kListLen] : 0.0f;
        uint32_t ek = (uint32_t)(e >> 32);
        uint32_t nx = wave_max_u32(lane64 < kRegBlock / 64 ? wave_next[lane64] : 0u);
#pragma unroll
        for (int r = 0; r <= kListLen; ++r) {
            const uint32_t m = wave_max_u32(ek);
            const int h = __ffsll((unsigned long long)__ballot(ek == m)) - 1;
            if (r < kListLen) {
                const uint32_t row = __builtin_amdgcn_readlane((uint32_t)e, h);
                const float val = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ev), h));
                if (lane64 == 0) {
                    ws->lists[r][my_slot] = (uint64_t)m << 32 | row;
                    if constexpr (SPEC)
                        ws->list_rec[r][my_slot] = val;
                }
            } else {
                nx = max(nx, m);
            }
            if (lane64 == h)
                ek = 0;
        }
        if (lane64 == 0)
            ws->lists[kListLen][my_slot] = (uint64_t)nx << 32;
    }
}

// Inclusive prefix sum over the 1024 threads of the workgroup (scan[] holds
// one word per wave).
__device__ inline int block_inclusive_scan(int v, int* scan)
{
    const int lane = threadIdx.x % 64, w = threadIdx.x / 64;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(v, d, 64);
        if (lane >= d)
            v += t;
    }
    __syncthreads();
    if (lane == 63)
        scan[w] = v;
    __syncthreads();
    int before = 0;
    for (int i = 0; i < w; ++i)
        before += scan[i];
    return v + before;
}

struct Entry {
    uint32_t key;
    int32_t row;
};

// a precedes b: larger logit, or equal logit and lower row
__device__ inline bool precedes(const Entry& a, const Entry& b)
{
    return a.key > b.key || (a.key == b.key && a.row < b.row);
}

// Bitonic sort of n = 2^p entries in LDS, best first (precedes), one entry
// per thread for the first n threads; every thread of the block calls it.
template <int N>
__device__ inline void bitonic_sort(Entry* e)
{
    const int tid = threadIdx.x;
    for (int size = 2; size <= N; size <<= 1) {
        for (int stride = size / 2; stride > 0; stride >>= 1) {
            if (tid < N) {
                const int partner = tid ^ stride;
                if (partner > tid) {
                    const bool up = (tid & size) == 0;  // this block sorts best-first
                    const Entry a = e[tid], b = e[partner];
                    if (up ? precedes(b, a) : precedes(a, b)) {
                        e[tid] = b;
                        e[partner] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
}

// The kk best entries of all V logits into sel[0 .. kk) in any order, by a
// radix select over the whole array (the path for inputs with so many equal
// logits that the candidate pool overflows).
__device__ inline void radix_select_all(const float* __restrict__ logits, int V, int kk, Entry* sel, int* hist,
                                        int* scan)
{
    __shared__ uint32_t s_prefix, s_mask;
    __shared__ int s_remaining, s_found, s_count;
    const int tid = threadIdx.x;
    if (tid == 0) {
        s_prefix = 0;
        s_mask = 0;
        s_remaining = kk;
        s_count = 0;
    }
    __syncthreads();
    // the kk-th largest key, 11 + 11 + 10 bits from the top
    constexpr int kShift[3] = {21, 10, 0};
    constexpr int kBits[3] = {11, 11, 10};
    int above_total = 0;  // keys strictly above the final prefix (same on all threads)
#pragma unroll
    for (int pass = 0; pass < 3; ++pass) {
        const int bins = 1 << kBits[pass];
        for (int b = tid; b < 2048; b += kSelectBlock)
            hist[b] = 0;
        __syncthreads();
        const uint32_t prefix = s_prefix, mask = s_mask;
        for (int e = tid; e < V; e += kSelectBlock) {
            const uint32_t key = order_key(logits[e]);
            if ((key & mask) == prefix)
                atomicAdd(&hist[(key >> kShift[pass]) & (bins - 1)], 1);
        }
        __syncthreads();
        // thread t owns bins (bins-1-2t, bins-2-2t): the highest bins first
        const int b_hi = bins - 1 - 2 * tid, b_lo = b_hi - 1;
        const int c_hi = b_hi >= 0 ? hist[b_hi] : 0;
        const int c_lo = b_lo >= 0 ? hist[b_lo] : 0;
        const int incl = block_inclusive_scan(c_hi + c_lo, scan);
        const int before = incl - c_hi - c_lo;  // keys in higher bins
        const int remaining = s_remaining;
        __syncthreads();
        if (b_hi >= 0 && before < remaining && remaining <= before + c_hi) {
            s_found = b_hi;
            s_remaining = remaining - before;
            scan[0] = before;
        } else if (b_lo >= 0 && before + c_hi < remaining && remaining <= before + c_hi + c_lo) {
            s_found = b_lo;
            s_remaining = remaining - before - c_hi;
            scan[0] = before + c_hi;
        }
        __syncthreads();
        above_total += scan[0];
        if (tid == 0) {
            s_prefix = prefix | ((uint32_t)s_found << kShift[pass]);
            s_mask = mask | ((uint32_t)(bins - 1) << kShift[pass]);
        }
        __syncthreads();
    }
    const uint32_t T = s_prefix;      // the kk-th largest key
    const int need_eq = s_remaining;  // entries equal to T to take, lowest rows first
    // keys above T: fewer than kk of them, appended in any order
    for (int e = tid; e < V; e += kSelectBlock) {
        const uint32_t key = order_key(logits[e]);
        if (key > T) {
            const int pos = atomicAdd(&s_count, 1);  // < kk by the selection
            if (pos < kHeadMaxK)
                sel[pos] = Entry{key, e};
        }
    }
    // keys equal to T: the need_eq lowest rows, by a scan in row order
    const int chunk = (V + kSelectBlock - 1) / kSelectBlock;
    const int e0 = min(V, tid * chunk), e1 = min(V, e0 + chunk);
    int n_eq = 0;
    for (int e = e0; e < e1; ++e)
        n_eq += order_key(logits[e]) == T;
    const int eq_before = block_inclusive_scan(n_eq, scan) - n_eq;
    int rank = eq_before;
    for (int e = e0; e < e1 && rank < need_eq; ++e) {
        if (order_key(logits[e]) == T) {
            if (above_total + rank < kHeadMaxK)
                sel[above_total + rank] = Entry{T, e};
            ++rank;
        }
    }
    __syncthreads();
}


// A pooled entry as one 64-bit code: the logit's key above, the row's
// complement below, so that a larger code precedes (larger logit, or equal
// logit and lower row) and one 64-bit compare orders two entries; code 0
// precedes nothing (key 0 marks "no element").
__device__ inline uint64_t pool_code(uint32_t key, int row)
{
    return (uint64_t)key << 32 | (uint32_t)~row;
}
__device__ inline Entry pool_entry(uint64_t code)
{
    return Entry{(uint32_t)(code >> 32), (int32_t)~(uint32_t)code};
}

// Append the lanes' entries with `take` set to the LDS pool: one LDS atomic
// per wave, positions by lane rank; entries past `cap` are counted, not kept.
// With `vals`, each entry's value goes to the same position there.
__device__ inline void pool_append(bool take, uint32_t key, int row, uint64_t* pool, int* count, int cap,
                                   float val = 0.0f, float* vals = nullptr)
{
    const uint64_t m = __ballot(take);
    if (m == 0)
        return;
    const int lane = threadIdx.x % 64;
    const int first = __ffsll((unsigned long long)m) - 1;
    int base = 0;
    if (lane == first)
        base = atomicAdd(count, __popcll(m));
    base = __builtin_amdgcn_readlane(base, first);
    const int pos = base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
    if (take && pos < cap) {
        pool[pos] = pool_code(key, row);
        if (vals)
            vals[pos] = val;
    }
}

constexpr int kScanUnroll = 16;      // logits per thread loaded before any is used (full scan)
constexpr int kMergeCap = 1024;      // pooled entries the selection ranks in LDS

// Rank selection of the kk best of n pooled entries into sel: the rank of
// an entry is the number of entries whose code is larger (a strict total
// order).  The count is bound by vector ALU work (16 waves on the CU's four
// SIMDs), so each comparison is one 64-bit compare and an add with carry,
// and the pool past n holds zero codes (kRankPad of them), so that reads
// need no clamp and counts no mask.  G threads count for each entry (G the
// largest power of two up to 64 with G n <= the block), thread p of the
// group over entries p, p + G, ..., and the G partial counts are summed
// across the group's lanes.
constexpr int kRankPad = 8;
__device__ inline void rank_pool(const uint64_t* pool, int n, int kk, Entry* sel, const float* vals = nullptr,
                                 float* sel_vals = nullptr)
{
    const int tid = threadIdx.x;
    int G = 1;
    while (G < 64 && 2 * G * n <= kSelectBlock)
        G *= 2;
    const int e = tid / G, p = tid % G;
    uint64_t me = 0;
    int rank = 0;
    if (e < n) {
        me = pool[e];
        for (int j = p; j < n; j += 8 * G) {  // eight LDS reads in flight, at most j + 7 G < n + 7 G
            uint64_t o[8];
#pragma unroll
            for (int t = 0; t < 8; ++t)
                o[t] = pool[j + t * G];
#pragma unroll
            for (int t = 0; t < 8; ++t)
                rank += o[t] > me;
        }
    }
    for (int d = 1; d < G; d <<= 1)  // G is the same in every thread
        rank += __shfl_xor(rank, d, 64);
    if (e < n && p == 0 && rank < kk) {
        sel[rank] = pool_entry(me);
        if (vals)
            sel_vals[rank] = vals[e];
    }
    __syncthreads();
}

// Candidate selection, gate and verification, one workgroup.  The
// approximate head left, per workgroup, its four largest logits, the largest
// key it did not list, and (SPEC) the listed rows recomputed with the FP32
// activations.  A lower bound L on the kk-th largest key: every wave takes
// the r = ceil(kk / 16) largest workgroup maxima it holds (distinct
// elements) and L is the least of those 16 r, so at least kk elements have
// keys >= L.  The listed entries at or above L are pooled and ranked; the
// result is exact
// when every key left out of the lists is below the kk-th selected key.
// Otherwise (many equal or clustered logits) the whole array is scanned:
// elements at or above L are pooled and ranked, or, past 1024 of them, a
// radix select picks the kk.  Then the gap and the gate; when verification
// runs, the candidates' recomputed logits come from the lists, or, after a
// whole-array selection, are computed here (one wave per row), and the token
// is the largest (ties: the lower row).
__global__ __launch_bounds__(kSelectBlock) void k_head_select(const float* __restrict__ logits, int V, int top_k,
                                                              float threshold, int n_approx, int spec,
                                                              const HeadWorkspace* __restrict__ ws,
                                                              const int8_t* __restrict__ Q,
                                                              const float* __restrict__ scale, int K,
                                                              const float* __restrict__ x,
                                                              int32_t* __restrict__ cand,
                                                              float* __restrict__ cand_logits,
                                                              int32_t* __restrict__ result)
{
    // pooled codes, zero past the count: n + 7 G <= kMergeCap + 7 for every
    // G rank_pool picks
    __shared__ uint64_t pool[kMergeCap + kRankPad];
    __shared__ float pool_rec[kMergeCap];
    __shared__ Entry sel[kHeadMaxK];
    __shared__ float sel_rec[kHeadMaxK];
    __shared__ int hist[2048];
    __shared__ int scan[kSelectBlock / 64];
    __shared__ uint32_t wave_low[kSelectBlock / 64], wave_next[kSelectBlock / 64];
    __shared__ int s_count;
    const int tid = threadIdx.x, lane = tid % 64, w = tid / 64;
    const int kk = V >= 2 ? max(top_k, 2) : 1;  // entries to select (the gap needs two)

    // this thread's workgroup list (spread so that each wave holds
    // ceil(n_approx / 16) of them), all loads at once
    const int b = lane * (kSelectBlock / 64) + w;
    uint64_t ent[kListLen + 1];
    float erec[kListLen];
#pragma unroll
    for (int i = 0; i <= kListLen; ++i)
        ent[i] = b < n_approx ? ws->lists[i][tid] : 0ull;
#pragma unroll
    for (int i = 0; i < kListLen; ++i)
        erec[i] = spec && b < n_approx ? ws->list_rec[i][tid] : 0.0f;
    uint32_t v = (uint32_t)(ent[0] >> 32);  // the workgroup's largest key
    for (int i = tid; i < kMergeCap + kRankPad; i += kSelectBlock)
        pool[i] = 0;
    if (tid == 0)
        s_count = 0;
    uint32_t low = 0xffffffffu;
    const int rounds = (kk + kSelectBlock / 64 - 1) / (kSelectBlock / 64);  // 16 rounds >= kk
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        if (r >= rounds)
            break;
        const uint32_t m = wave_max_u32(v);
        low = min(low, m);
        const uint64_t holders = __ballot(v == m);
        if (lane == __ffsll((unsigned long long)holders) - 1)
            v = 0;
    }
    const uint32_t nmax = wave_max_u32((uint32_t)(ent[kListLen] >> 32));
    if (lane == 0) {
        wave_low[w] = low;
        wave_next[w] = nmax;
    }
    __syncthreads();
    uint32_t L = wave_low[0], max_next = wave_next[0];
#pragma unroll
    for (int i = 1; i < kSelectBlock / 64; ++i) {
        L = min(L, wave_low[i]);
        max_next = max(max_next, wave_next[i]);
    }
    L = max(L, 1u);  // key 0 marks "no element"
    {
        // the listed entries at or above L, one LDS atomic per wave: the
        // lane's count in three ballots, its offset the count of the lanes
        // below it
        int cnt = 0;
#pragma unroll
        for (int i = 0; i < kListLen; ++i)
            cnt += (uint32_t)(ent[i] >> 32) >= L;
        const uint64_t b0 = __ballot(cnt & 1), b1 = __ballot(cnt & 2), b2 = __ballot(cnt & 4);
        const int total = __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2);
        if (total > 0) {
            auto below = [&](uint64_t m) {
                return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
            };
            int base = 0;
            if (lane == 0)
                base = atomicAdd(&s_count, total);
            int pos = __builtin_amdgcn_readlane(base, 0) + below(b0) + 2 * below(b1) + 4 * below(b2);
#pragma unroll
            for (int i = 0; i < kListLen; ++i) {
                const uint32_t k = (uint32_t)(ent[i] >> 32);
                if (k >= L) {
                    if (pos < kMergeCap) {
                        pool[pos] = pool_code(k, (int32_t)(uint32_t)ent[i]);
                        pool_rec[pos] = erec[i];
                    }
                    ++pos;
                }
            }
        }
    }
    __syncthreads();
    int n_pool = s_count;
    bool exact = n_pool <= kMergeCap;
    if (exact) {
        rank_pool(pool, n_pool, kk, sel, pool_rec, sel_rec);
        exact = n_pool >= kk && max_next < sel[kk - 1].key;
    }
    if (!exact) {
        // the lists may miss elements: every logit at or above L
        __syncthreads();
        for (int i = tid; i < kMergeCap + kRankPad; i += kSelectBlock)
            pool[i] = 0;
        if (tid == 0)
            s_count = 0;
        __syncthreads();
        for (int e0 = tid; e0 < V; e0 += kScanUnroll * kSelectBlock) {
            uint32_t g[kScanUnroll];  // all loads of the batch in flight at once
#pragma unroll
            for (int u = 0; u < kScanUnroll; ++u) {
                const int e = e0 + u * kSelectBlock;
                g[u] = e < V ? order_key(logits[e]) : 0u;
            }
#pragma unroll
            for (int u = 0; u < kScanUnroll; ++u)
                pool_append(g[u] >= L, g[u], e0 + u * kSelectBlock, pool, &s_count, kMergeCap);
        }
        __syncthreads();
        n_pool = s_count;
        if (n_pool <= kMergeCap) {
            rank_pool(pool, n_pool, kk, sel);
        } else {
            radix_select_all(logits, V, kk, sel, hist, scan);
            if (tid < kHeadMaxK && tid >= kk)
                sel[tid] = Entry{0u, 0x7fffffff};
            __syncthreads();
            bitonic_sort<kHeadMaxK>(sel);
        }
    }

    const float l1 = key_value(sel[0].key);
    const float gap = V >= 2 ? l1 - key_value(sel[1].key) : __builtin_inff();
    const bool verify = gap < threshold;
    if (tid < top_k)
        cand[tid] = sel[tid].row;
    if (!verify) {
        if (tid < top_k)
            cand_logits[tid] = key_value(sel[tid].key);
        if (tid == 0) {
            result[0] = sel[0].row;
            result[1] = 0;
        }
        return;
    }
    if (!(exact && spec)) {
        // wave w recomputes candidates w, w + 16, w + 32, w + 48
        for (int i = w; i < top_k; i += kSelectBlock / 64) {
            const float r = recompute_row(Q, scale, K, x, sel[i].row);
            if (lane == 0)
                sel_rec[i] = r;
        }
        __syncthreads();
    }
    if (tid < top_k)
        cand_logits[tid] = sel_rec[tid];
    if (w == 0) {
        // the largest recomputed logit, ties to the lower row: wave maximum
        // of the key, then the least row holding it
        const uint32_t key = lane < top_k ? order_key(sel_rec[lane]) : 0u;
        const uint32_t top = wave_max_u32(key);
        const uint32_t row = key == top ? (uint32_t)sel[lane].row : 0xffffffffu;
        const uint32_t least = ~wave_max_u32(~row);
        if (lane == 0) {
            result[0] = (int32_t)least;
            result[1] = 1;
        }
    }
}

}  // namespace spk
