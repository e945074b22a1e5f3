// Dense continuous-input projection with weight-only INT8 storage (gfx950).
//
// The continuous-input projections of the model (attention query/key/value
// and output, feed-forward up, vocabulary head) keep row-major INT8 weights
// Q[m*K + k] with one FP32 scale s_m per output channel.  Each weight is
// converted to FP32, multiplied by the FP32 activation, the products are
// accumulated in FP32, and the row scale is applied once (paper Sec. 2.3,
// end of "Quantization and Accumulation"; Fig. "execution", lower path):
//
//     y[b][m] = s_m * sum_k float(Q[m][k]) * x[b][k]
//
// At decode batch sizes this reads every weight byte once, so it is an HBM
// stream, not a matrix-core contraction.  Work split: a workgroup of 256
// threads is 16 lane groups of 16 lanes; group g of workgroup w owns rows
// w * 16 * RPG + g + 16 r (r < RPG), so the 16 groups read 16 consecutive
// rows at a time.  Lane l of a group takes the V-byte chunks c = l + 16 j
// (j < ceil(K / (16 V))) of each of its rows.  Each lane walks its (row,
// chunk) items through a ring of U buffer loads (positions past the matrix
// read as zero), converts each weight byte with one sign-extending SDWA
// convert, and accumulates with FMAs, one FP32 accumulator per batch row;
// the activations (BC batch rows) and the workgroup's row scales are staged
// in LDS once per workgroup.  At
// the end of a row the 16 lanes are summed with cross-lane shuffles and
// lane 0 writes y = sum * s_m.
//
// Summation order, for the test tolerance: per lane one FMA chain over its
// chunks of the row (at most ceil(K / 16) products), then a 4-level tree
// over the 16 lanes, then one multiply by s_m.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "buffer.hpp"

namespace spk {

constexpr int kDenseBlock = 256;
constexpr int kDenseLanes = 16;                          // lanes per row
constexpr int kDenseGroups = kDenseBlock / kDenseLanes;  // rows in flight per workgroup
constexpr int kDenseMaxLdsFloats = 16384;  // dynamic LDS of one workgroup: 64 KB

// byte BYTE of d, sign-extended, as FP32 (one SDWA convert)
template <int BYTE>
__device__ inline float cvt_i8(uint32_t d)
{
    float f;
    if constexpr (BYTE == 0)
        asm("v_cvt_f32_i32_sdwa %0, sext(%1) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0" : "=v"(f) : "v"(d));
    else if constexpr (BYTE == 1)
        asm("v_cvt_f32_i32_sdwa %0, sext(%1) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1" : "=v"(f) : "v"(d));
    else if constexpr (BYTE == 2)
        asm("v_cvt_f32_i32_sdwa %0, sext(%1) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2" : "=v"(f) : "v"(d));
    else
        asm("v_cvt_f32_i32_sdwa %0, sext(%1) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3" : "=v"(f) : "v"(d));
    return f;
}

// V weight bytes of one chunk, loaded through a buffer resource (nontemporal).
template <int V>
struct DenseChunk;
template <>
struct DenseChunk<16> {
    u32x4 v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2); }
    __device__ uint32_t word(int i) const { return v[i]; }
};
template <>
struct DenseChunk<4> {
    uint32_t v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 2); }
    __device__ uint32_t word(int) const { return v; }
};
template <>
struct DenseChunk<1> {
    uint32_t v;
    __device__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = __builtin_amdgcn_raw_buffer_load_b8(r, off, 0, 2); }
    __device__ uint32_t word(int) const { return v; }
};

// acc[b] += w[t] * x[b][k0 + t] for t = 0..V-1, in that order.
template <int V, int BC>
__device__ inline void dense_fma(const DenseChunk<V>& q, const float* xs, int x_pitch, int k0, float (&acc)[BC])
{
    if constexpr (V == 1) {
        const float w = cvt_i8<0>(q.word(0));
#pragma unroll
        for (int b = 0; b < BC; ++b)
            acc[b] = __builtin_fmaf(w, xs[b * x_pitch + k0], acc[b]);
    } else {
        float w[V];
#pragma unroll
        for (int i = 0; i < V / 4; ++i) {
            const uint32_t d = q.word(i);
            w[4 * i + 0] = cvt_i8<0>(d);
            w[4 * i + 1] = cvt_i8<1>(d);
            w[4 * i + 2] = cvt_i8<2>(d);
            w[4 * i + 3] = cvt_i8<3>(d);
        }
#pragma unroll
        for (int b = 0; b < BC; ++b) {
            const float* xb = xs + b * x_pitch + k0;
#pragma unroll
            for (int t = 0; t < V; t += 4) {
                const f32x4 x4 = *reinterpret_cast<const f32x4*>(xb + t);
                acc[b] = __builtin_fmaf(w[t + 0], x4.x, acc[b]);
                acc[b] = __builtin_fmaf(w[t + 1], x4.y, acc[b]);
                acc[b] = __builtin_fmaf(w[t + 2], x4.z, acc[b]);
                acc[b] = __builtin_fmaf(w[t + 3], x4.w, acc[b]);
            }
        }
    }
}

// LDS floats per staged activation row: K, plus V zeros that lanes with no
// chunk left in a row read (their weights are zero too), rounded up to a
// multiple of 4.
__host__ __device__ constexpr int dense_x_pitch(int K, int V) { return (K + V + 3) / 4 * 4; }

// Dynamic LDS floats of a launch: BC activation rows and the scales of the
// workgroup's rows (read from LDS so that no global load sits between the
// ring's loads and their waits).
__host__ __device__ constexpr int dense_lds_floats(int K, int V, int bc, int rpg)
{
    return bc * dense_x_pitch(K, V) + kDenseGroups * rpg;
}

// Walks (row r, chunk j) items of one lane in order: item i is r = i / n_pl,
// j = i % n_pl.
struct DenseCursor {
    int r, j;
    __device__ void step(int n_pl)
    {
        if (++j == n_pl) {
            j = 0;
            ++r;
        }
    }
};

// y[b][m] for b < B (B <= BC), rows m of this workgroup.  Needs M * K below
// 2^31 (one buffer resource), dense_lds_floats(K, V, BC,
// rpg) floats of dynamic LDS, and a Q base aligned to V bytes.
template <int V, int BC, int U>
__global__ __launch_bounds__(kDenseBlock) void k_dense(const int8_t* __restrict__ Q, const float* __restrict__ scale,
                                                       int K, int M, const float* __restrict__ x, int B,
                                                       float* __restrict__ y, int rpg)
{
    extern __shared__ __align__(16) float xs[];
    const int g = threadIdx.x / kDenseLanes;
    const int l = threadIdx.x % kDenseLanes;
    const int row0 = blockIdx.x * kDenseGroups * rpg + g;  // the group's rows: row0 + 16 r
    const int n_chunks = K / V;
    const int n_pl = (n_chunks + kDenseLanes - 1) / kDenseLanes;  // chunks per lane per row
    const int n_items = rpg * n_pl;
    const __amdgpu_buffer_rsrc_t res = weight_resource(Q, (int64_t)M * K);
    auto offset_of = [&](const DenseCursor& p) -> uint32_t {
        const int m = row0 + kDenseGroups * p.r;
        const int c = l + kDenseLanes * p.j;
        const bool ok = p.r < rpg && m < M && c < n_chunks;
        return ok ? (uint32_t)m * (uint32_t)K + (uint32_t)(c * V) : kOutOfRange;
    };

    // the first round of weight loads goes out before the activations are staged
    DenseChunk<V> slot[U];
    DenseCursor ahead{0, 0};
#pragma unroll
    for (int u = 0; u < U; ++u) {
        slot[u].load(res, offset_of(ahead));
        ahead.step(n_pl);
    }
    const int pitch = dense_x_pitch(K, V);
    for (int e = threadIdx.x; e < BC * pitch; e += kDenseBlock) {
        const int b = e / pitch, k = e - b * pitch;
        xs[e] = (b < B && k < K) ? x[(int64_t)b * K + k] : 0.0f;
    }
    float* ss = xs + BC * pitch;  // scales of rows blockIdx.x * 16 * rpg + e
    for (int e = threadIdx.x; e < kDenseGroups * rpg; e += kDenseBlock) {
        const int m = blockIdx.x * kDenseGroups * rpg + e;
        ss[e] = m < M ? scale[m] : 0.0f;
    }
    __syncthreads();

    float acc[BC];
#pragma unroll
    for (int b = 0; b < BC; ++b)
        acc[b] = 0.0f;
    DenseCursor cur{0, 0};
    for (int i0 = 0; i0 < n_items; i0 += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = min(l + kDenseLanes * cur.j, n_chunks);  // n_chunks: the zero tail
            dense_fma<V, BC>(slot[u], xs, pitch, c * V, acc);
            slot[u].load(res, offset_of(ahead));
            ahead.step(n_pl);
            __builtin_amdgcn_sched_barrier(0);
            if (cur.j == n_pl - 1) {  // end of a row (uniform over the wave)
#pragma unroll
                for (int b = 0; b < BC; ++b) {
                    float v = acc[b];
                    v += __shfl_xor(v, 8, 64);
                    v += __shfl_xor(v, 4, 64);
                    v += __shfl_xor(v, 2, 64);
                    v += __shfl_xor(v, 1, 64);
                    acc[b] = v;
                }
                const int m = row0 + kDenseGroups * cur.r;
                if (l == 0 && cur.r < rpg && m < M) {
                    const float s = ss[g + kDenseGroups * cur.r];
#pragma unroll
                    for (int b = 0; b < BC; ++b)
                        if (b < B)
                            y[(int64_t)b * M + m] = acc[b] * s;
                }
#pragma unroll
                for (int b = 0; b < BC; ++b)
                    acc[b] = 0.0f;
            }
            cur.step(n_pl);
        }
    }
}


// ---------------------------------------------------------------------------
// Register-resident variant for K <= 512 * NPL with K % 16 == 0 and a 16-byte
// aligned Q (the model's continuous projections all have K = 1536, NPL = 3).
//
// A lane group is 32 lanes (two per wave).  Lane l always covers the same
// 16-byte chunks c = l + 32 j (j < NPL) of a row, so its slice of the BC
// activation rows is loaded into registers once and the inner loop touches
// no LDS.  Group q of the grid's Gq groups takes rows m = q + Gq r
// (r = 0, 1, ...): at each step the whole grid reads one contiguous band
// of rows.  A lane keeps a ring of U rows of loads (U * NPL 16-byte loads)
// in flight.  A row's 32 partial sums are combined by a 5-level tree (DPP
// within 16 lanes, one swizzle across the halves); the sum for the group's
// r-th row is parked in lane r % 32, and every 32 rows the parked sums are
// scaled (each lane has its row's scale loaded a block ahead) and go out in
// one scattered store instead of 32 single-lane ones.
//
// Summation order: per lane one FMA chain over its NPL chunks (j, then byte
// order), then the 5-level tree, then one multiply by the row scale; it
// depends on K only, not on B, the batch split or the grid.
// ---------------------------------------------------------------------------
constexpr int kRegLanes = 32;
constexpr int kRegBlock = 256;
constexpr int kRegGroups = kRegBlock / kRegLanes;  // 8 groups per workgroup

template <int CTRL>
__device__ inline float add_dpp(float v)
{
    const int moved = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false);
    return v + __builtin_bit_cast(float, moved);
}

// Sum over the 32 lanes of a group; every lane of the group gets the total.
__device__ inline float group32_sum(float v)
{
    v = add_dpp<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
    v = add_dpp<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
    v = add_dpp<0x141>(v);  // row_half_mirror: the other quad of 8 lanes
    v = add_dpp<0x140>(v);  // row_mirror: the other 8 lanes of 16
    const int other = __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F);  // lane ^ 16
    return v + __builtin_bit_cast(float, other);
}

template <int NPL, int BC, int U>
__global__ __launch_bounds__(kRegBlock) void k_dense_reg(const int8_t* __restrict__ Q, const float* __restrict__ scale,
                                                         int K, int M, const float* __restrict__ x, int B,
                                                         float* __restrict__ y)
{
    const int l = threadIdx.x % kRegLanes;
    const int q = blockIdx.x * kRegGroups + threadIdx.x / kRegLanes;  // group id
    const int Gq = gridDim.x * kRegGroups;
    const int q_wave = q & ~1;  // first group of the wave: the step count is the wave's
    const int n_steps = __builtin_amdgcn_readfirstlane(q_wave < M ? (M - q_wave + Gq - 1) / Gq : 0);
    const int n_chunks = K / 16;
    const __amdgpu_buffer_rsrc_t qres = weight_resource(Q, (int64_t)M * K);
    const __amdgpu_buffer_rsrc_t sres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(scale), 0, M * 4, kBufferFlags);

    // Byte offset of each chunk within a row.  A lane past the end of the row
    // re-reads chunk 0 (bytes the group loads anyway) and multiplies it by
    // its zero activations.
    uint32_t chunk_off[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int c = l + kRegLanes * j;
        chunk_off[j] = c < n_chunks ? (uint32_t)(c * 16) : 0u;
    }
    // row offset, or kOutOfRange past the rows (kOutOfRange + chunk offset < 2^32
    // stays past the resource)
    auto row_base = [&](int r) -> uint32_t {
        const int m = q + Gq * r;
        return r < n_steps && m < M ? (uint32_t)m * (uint32_t)K : kOutOfRange;
    };

    // this lane's activations, x[b][c*16 + t] for its chunks c (zeros past K
    // and B), are loaded before the ring so that waiting for them drains nothing
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(x), 0, B * K * 4, kBufferFlags);
    float xr[BC][NPL][16];
#pragma unroll
    for (int b = 0; b < BC; ++b)
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int c = l + kRegLanes * j;
            const uint32_t base = (b < B && c < n_chunks) ? (uint32_t)(b * K + c * 16) * 4u : kOutOfRange;
#pragma unroll
            for (int t = 0; t < 16; ++t)
                xr[b][j][t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, base + 4 * t, 0, 0));
        }

    // Scale of the row of step (32-row block start) + l, read at the block's
    // flush; the first block's goes out before the ring, the next block's at
    // each flush, so no flush waits on a fresh load.
    auto scale_of_step = [&](int rr) -> float {
        const int m = q + Gq * rr;
        const uint32_t off = rr < n_steps && m < M ? (uint32_t)m * 4u : kOutOfRange;
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sres, off, 0, 0));
    };
    float sc = scale_of_step(l);

    u32x4 slot[U][NPL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t base = row_base(u);
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            slot[u][j] = __builtin_amdgcn_raw_buffer_load_b128(qres, base + chunk_off[j], 0, 2);
    }

    float parked[BC];  // lane i holds the sum of the group's step r with r % 32 == i
#pragma unroll
    for (int b = 0; b < BC; ++b)
        parked[b] = 0.0f;
    for (int r0 = 0; r0 < n_steps; r0 += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = r0 + u;
            float acc[BC];
#pragma unroll
            for (int b = 0; b < BC; ++b)
                acc[b] = 0.0f;
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t d = slot[u][j][i];
                    const float w0 = cvt_i8<0>(d), w1 = cvt_i8<1>(d), w2 = cvt_i8<2>(d), w3 = cvt_i8<3>(d);
#pragma unroll
                    for (int b = 0; b < BC; ++b) {
                        acc[b] = __builtin_fmaf(w0, xr[b][j][4 * i + 0], acc[b]);
                        acc[b] = __builtin_fmaf(w1, xr[b][j][4 * i + 1], acc[b]);
                        acc[b] = __builtin_fmaf(w2, xr[b][j][4 * i + 2], acc[b]);
                        acc[b] = __builtin_fmaf(w3, xr[b][j][4 * i + 3], acc[b]);
                    }
                }
            }
            {  // refill the slot with row r + U
                const uint32_t base = row_base(r + U);
#pragma unroll
                for (int j = 0; j < NPL; ++j)
                    slot[u][j] = __builtin_amdgcn_raw_buffer_load_b128(qres, base + chunk_off[j], 0, 2);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int b = 0; b < BC; ++b) {
                const float tot = group32_sum(acc[b]);
                if (l == (r & 31))
                    parked[b] = tot;
            }
            // Flush the parked rows of steps r - r % 32 .. r: scale and store.
            if (r < n_steps && ((r & 31) == 31 || r == n_steps - 1)) {
                const int rr = (r & ~31) + l;
                const int m = q + Gq * rr;
                if (rr <= r && m < M) {
#pragma unroll
                    for (int b = 0; b < BC; ++b)
                        if (b < B)
                            y[(int64_t)b * M + m] = parked[b] * sc;
                }
                sc = scale_of_step((r & ~31) + 32 + l);
            }
        }
    }
}

}  // namespace spk
