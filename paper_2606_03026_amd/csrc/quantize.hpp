// Symmetric per-output-channel INT8 quantization and export (gfx950).
//
// For a weight matrix W [M][K] (row m = output channel m), paper Sec. 2.3:
//
//     s_m     = max(max_k |W[m][k]|, 1e-8) / 127
//     Q[m][k] = clip(round(W[m][k] / s_m), -127, 127)
//
// in binary32: the maximum is exact, both divisions are correctly rounded
// (v_div_scale / v_div_fmas / v_div_fixup, no reciprocal approximation),
// and round() is v_rndne (ties to even).  Q is written row-major (the dense
// continuous-input layout) or column-major (W_cm[k][m] = Q[m][k], the
// spike-gated layout, Sec. 2.2).
//
// Row-major output with rows of at most 4096 values (K % 4 == 0, aligned):
// one pass, k_quant_rows -- one wave per row holds the row in registers,
// reduces its maximum over the wave, writes s and the row of Q.  Otherwise
// two passes, both bound by HBM: k_quant_scale reads each row once (one wave
// per row, a max-reduction over the wave) and writes s; k_quant_tile reads W
// again in 64 x 64 tiles, quantizes, and writes Q.  For the column-major
// layout the tile is transposed through LDS so that both the reads (along k)
// and the writes (along m) are contiguous.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spk {

constexpr int kQuantBlock = 256;
constexpr int kQuantTile = 64;  // rows (m) and columns (k) of a tile

// one wave per row: s[m] from the row's largest magnitude.  VEC (K % 4 == 0,
// W 16-byte aligned): 16-byte loads; either way 8 loads per lane are in
// flight before any is used.
template <bool VEC>
__global__ __launch_bounds__(kQuantBlock) void k_quant_scale(const float* __restrict__ W, int M, int K,
                                                             float* __restrict__ scale)
{
    const int lane = threadIdx.x % 64;
    const int m = blockIdx.x * (kQuantBlock / 64) + threadIdx.x / 64;
    if (m >= M)
        return;
    const float* row = W + (int64_t)m * K;
    constexpr int kBatch = 8;
    float amax = 0.0f;
    if constexpr (VEC) {
        const float4* row4 = reinterpret_cast<const float4*>(row);
        const int n4 = K / 4;
        for (int c0 = lane; c0 < n4; c0 += 64 * kBatch) {
            float4 v[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int c = c0 + 64 * u;
                v[u] = c < n4 ? row4[c] : float4{0.0f, 0.0f, 0.0f, 0.0f};
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[u].x), fabsf(v[u].y)), fmaxf(fabsf(v[u].z), fabsf(v[u].w))));
        }
    } else {
        for (int k0 = lane; k0 < K; k0 += 64 * kBatch) {
            float v[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int k = k0 + 64 * u;
                v[u] = k < K ? row[k] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                amax = fmaxf(amax, fabsf(v[u]));
        }
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1)
        amax = fmaxf(amax, __shfl_xor(amax, d, 64));
    if (lane == 0)
        scale[m] = __fdiv_rn(fmaxf(amax, 1e-8f), 127.0f);
}

__device__ inline int8_t quantize_one(float w, float s)
{
    const float r = __builtin_rintf(__fdiv_rn(w, s));
    return (int8_t)fminf(fmaxf(r, -127.0f), 127.0f);
}

// One wave per row, the row in registers: lane l holds the float4 chunks
// l + 64 j (j < NV) of its row, so K <= 256 NV.  Needs K % 4 == 0, W 16-byte
// and Q 4-byte aligned (host-checked).
constexpr int kQuantRowsMaxK = 4096;
template <int NV>
__global__ __launch_bounds__(kQuantBlock) void k_quant_rows(const float* __restrict__ W, int M, int K,
                                                            int8_t* __restrict__ Q, float* __restrict__ scale)
{
    const int lane = threadIdx.x % 64;
    const int m = blockIdx.x * (kQuantBlock / 64) + threadIdx.x / 64;
    if (m >= M)
        return;
    const int n4 = K / 4;
    const float4* row = reinterpret_cast<const float4*>(W + (int64_t)m * K);
    float4 w[NV];
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int c = lane + 64 * j;
        w[j] = c < n4 ? row[c] : float4{0.0f, 0.0f, 0.0f, 0.0f};
    }
#pragma unroll
    for (int j = 0; j < NV; ++j)
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(w[j].x), fabsf(w[j].y)), fmaxf(fabsf(w[j].z), fabsf(w[j].w))));
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1)
        amax = fmaxf(amax, __shfl_xor(amax, d, 64));
    const float s = __fdiv_rn(fmaxf(amax, 1e-8f), 127.0f);
    if (lane == 0)
        scale[m] = s;
    uint32_t* dst = reinterpret_cast<uint32_t*>(Q + (int64_t)m * K);
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int c = lane + 64 * j;
        if (c < n4)
            dst[c] = (uint32_t)(uint8_t)quantize_one(w[j].x, s) | (uint32_t)(uint8_t)quantize_one(w[j].y, s) << 8 |
                     (uint32_t)(uint8_t)quantize_one(w[j].z, s) << 16 |
                     (uint32_t)(uint8_t)quantize_one(w[j].w, s) << 24;
    }
}

// One 64 x 64 tile (rows m0.., columns k0..) per workgroup.  Each thread
// takes 4 consecutive columns of 4 rows.  COL: write W_cm[k][m] through an
// LDS transpose, 4 consecutive m per thread.  VEC (host-checked: K % 4 == 0,
// W 16-byte aligned, Q 4-byte aligned, and M % 4 == 0 for COL): 16-byte
// loads of W and 4-byte stores of Q; otherwise element by element.
template <bool COL, bool VEC>
__global__ __launch_bounds__(kQuantBlock) void k_quant_tile(const float* __restrict__ W, const float* __restrict__ scale,
                                                            int M, int K, int8_t* __restrict__ Q, int tiles_k)
{
    __shared__ __align__(16) int8_t tile[kQuantTile][kQuantTile + 4];  // [k][m] for COL
    const int m0 = (blockIdx.x / tiles_k) * kQuantTile;
    const int k0 = (blockIdx.x % tiles_k) * kQuantTile;
    const int c4 = (threadIdx.x % 16) * 4;  // first of the thread's 4 columns
    const int r0 = threadIdx.x / 16;        // rows r0 + 16 i
#pragma unroll
    for (int i = 0; i < kQuantTile / 16; ++i) {
        const int r = r0 + 16 * i;
        const int m = m0 + r, k = k0 + c4;
        int8_t q[4] = {0, 0, 0, 0};
        if (m < M) {
            const float s = scale[m];
            const float* src = W + (int64_t)m * K + k;
            if (VEC && k + 3 < K) {
                const float4 w = *reinterpret_cast<const float4*>(src);
                q[0] = quantize_one(w.x, s);
                q[1] = quantize_one(w.y, s);
                q[2] = quantize_one(w.z, s);
                q[3] = quantize_one(w.w, s);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (k + j < K)
                        q[j] = quantize_one(src[j], s);
            }
        }
        if constexpr (COL) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                tile[c4 + j][r] = q[j];
        } else if (m < M) {
            int8_t* dst = Q + (int64_t)m * K + k;
            if (VEC && k + 3 < K) {
                *reinterpret_cast<uint32_t*>(dst) = (uint32_t)(uint8_t)q[0] | (uint32_t)(uint8_t)q[1] << 8 |
                                                    (uint32_t)(uint8_t)q[2] << 16 | (uint32_t)(uint8_t)q[3] << 24;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (k + j < K)
                        dst[j] = q[j];
            }
        }
    }
    if constexpr (COL) {
        __syncthreads();
        // thread: 4 consecutive m (mm .. mm + 3) of the tile's columns kk
#pragma unroll
        for (int i = 0; i < kQuantTile / 16; ++i) {
            const int kk = r0 + 16 * i;
            const int k = k0 + kk, m = m0 + c4;
            if (k >= K)
                continue;
            int8_t* dst = Q + (int64_t)k * M + m;
            if (VEC && m + 3 < M) {
                *reinterpret_cast<uint32_t*>(dst) = *reinterpret_cast<const uint32_t*>(&tile[kk][c4]);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (m + j < M)
                        dst[j] = tile[kk][c4 + j];
            }
        }
    }
}

}  // namespace spk
