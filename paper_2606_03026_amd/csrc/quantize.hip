// Host side of the INT8 quantizer/exporter (C ABI in include/quantize.h):
// validation and the launches.  No allocation, no synchronisation.
#include "quantize.h"

#include <hip/hip_runtime.h>

#include <cstdint>

#include "errors.hpp"
#include "quantize.hpp"

namespace {

using spk::fail;
using spk::hip_fail;

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

template <bool COL>
void launch_tile(bool vec, dim3 grid, hipStream_t st, const float* W, const float* scale, int M, int K, int8_t* Q,
                 int tiles_k)
{
    if (vec)
        hipLaunchKernelGGL((spk::k_quant_tile<COL, true>), grid, dim3(spk::kQuantBlock), 0, st, W, scale, M, K, Q,
                           tiles_k);
    else
        hipLaunchKernelGGL((spk::k_quant_tile<COL, false>), grid, dim3(spk::kQuantBlock), 0, st, W, scale, M, K, Q,
                           tiles_k);
}

}  // namespace

extern "C" {

int spike_quantize_int8(const float* W, int32_t M, int32_t K, int32_t layout, int8_t* Q, float* scale, void* stream)
{
    spk::last_error.clear();
    if (M < 1 || M > (1 << 24))
        return fail(SPIKE_EINVAL, "M = %d outside [1, 2^24]", M);
    if (K < 1 || K > (1 << 24))
        return fail(SPIKE_EINVAL, "K = %d outside [1, 2^24]", K);
    if ((int64_t)M * K > (int64_t)1 << 31)
        return fail(SPIKE_EINVAL, "M * K = %lld exceeds 2^31", (long long)M * K);
    if (layout != SPIKE_LAYOUT_ROW_MAJOR && layout != SPIKE_LAYOUT_COL_MAJOR)
        return fail(SPIKE_EINVAL, "layout %d is not SPIKE_LAYOUT_ROW_MAJOR or SPIKE_LAYOUT_COL_MAJOR", layout);
    if (!W || !Q || !scale)
        return fail(SPIKE_EINVAL, "null pointer (W %p, Q %p, scale %p)", (const void*)W, (const void*)Q,
                    (const void*)scale);
    if (!aligned(W, 4) || !aligned(scale, 4))
        return fail(SPIKE_EINVAL, "W and scale must be 4-byte aligned");
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const int rows_per_block = spk::kQuantBlock / 64;
    const dim3 row_grid((M + rows_per_block - 1) / rows_per_block);
    if (layout == SPIKE_LAYOUT_ROW_MAJOR && K % 4 == 0 && K <= spk::kQuantRowsMaxK && aligned(W, 16) &&
        aligned(Q, 4)) {
        // one pass: each row read once, held in registers
        const int nv = (K + 255) / 256;
        if (nv <= 2)
            hipLaunchKernelGGL(spk::k_quant_rows<2>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, Q, scale);
        else if (nv <= 4)
            hipLaunchKernelGGL(spk::k_quant_rows<4>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, Q, scale);
        else if (nv <= 6)
            hipLaunchKernelGGL(spk::k_quant_rows<6>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, Q, scale);
        else if (nv <= 8)
            hipLaunchKernelGGL(spk::k_quant_rows<8>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, Q, scale);
        else
            hipLaunchKernelGGL(spk::k_quant_rows<16>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, Q, scale);
        const hipError_t e = hipGetLastError();
        return e == hipSuccess ? SPIKE_OK : hip_fail(e, "quantizer launch");
    }
    if (K % 4 == 0 && aligned(W, 16))
        hipLaunchKernelGGL(spk::k_quant_scale<true>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, scale);
    else
        hipLaunchKernelGGL(spk::k_quant_scale<false>, row_grid, dim3(spk::kQuantBlock), 0, st, W, M, K, scale);
    const int tiles_m = (M + spk::kQuantTile - 1) / spk::kQuantTile;
    const int tiles_k = (K + spk::kQuantTile - 1) / spk::kQuantTile;
    const dim3 grid((unsigned)((int64_t)tiles_m * tiles_k));
    const bool col = layout == SPIKE_LAYOUT_COL_MAJOR;
    const bool vec = K % 4 == 0 && aligned(W, 16) && aligned(Q, 4) && (!col || M % 4 == 0);
    if (col)
        launch_tile<true>(vec, grid, st, W, scale, M, K, Q, tiles_k);
    else
        launch_tile<false>(vec, grid, st, W, scale, M, K, Q, tiles_k);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "quantizer launch");
    return SPIKE_OK;
}

int spike_check_scale_shape(int32_t M, int32_t K, int32_t group, int32_t scale_rows, int32_t scale_cols)
{
    spk::last_error.clear();
    if (M < 1 || K < 1 || group < 1)
        return fail(SPIKE_EINVAL, "M = %d, K = %d and group = %d must be positive", M, K, group);
    const int64_t want_cols = ((int64_t)K + group - 1) / group;
    if (scale_rows == M && scale_cols == want_cols)
        return SPIKE_OK;
    const int64_t t_cols = ((int64_t)M + group - 1) / group;
    if (scale_rows == K && scale_cols == t_cols && !(M == K))
        return fail(SPIKE_EINVAL,
                    "scale shape [%d][%d] is that of the transposed [%d][%d] matrix: the scales were taken along "
                    "the input axis; a [%d][%d] weight with group %d needs [%d][%lld]",
                    scale_rows, scale_cols, K, M, M, K, group, M, (long long)want_cols);
    return fail(SPIKE_EINVAL, "scale shape [%d][%d] does not match a [%d][%d] weight with group %d (needs [%d][%lld])",
                scale_rows, scale_cols, M, K, group, M, (long long)want_cols);
}

}  // extern "C"
