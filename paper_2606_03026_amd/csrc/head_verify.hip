// Host side of the output-head candidate verification (C ABI in
// include/head_verify.h): validation and the launches.
#include "head_verify.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "errors.hpp"
#include "head.hpp"

namespace {

using spk::fail;
using spk::hip_fail;

using ApproxFn = void (*)(const int8_t*, const float*, int, int, const float*, float*, spk::HeadWorkspace*);

template <int NPL, bool SPEC>
ApproxFn approx_fn()
{
    return spk::k_head_approx<NPL, (NPL >= 4 ? 2 : 8 / NPL), SPEC>;
}

template <bool SPEC>
ApproxFn pick_approx(int npl)
{
    switch (npl) {
    case 1: return approx_fn<1, SPEC>();
    case 2: return approx_fn<2, SPEC>();
    case 3: return approx_fn<3, SPEC>();
    case 4: return approx_fn<4, SPEC>();
    case 5: return approx_fn<5, SPEC>();
    case 6: return approx_fn<6, SPEC>();
    case 7: return approx_fn<7, SPEC>();
    default: return approx_fn<8, SPEC>();
    }
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace

extern "C" {

int64_t head_verify_workspace_bytes(void) { return (int64_t)sizeof(spk::HeadWorkspace); }

int head_verify_forward(const int8_t* Q, const float* scale, int32_t K, int32_t V, const float* x, int32_t top_k,
                        float threshold, float* logits, int32_t* cand, float* cand_logits, int32_t* result,
                        void* workspace, void* stream)
{
    spk::last_error.clear();
    if (K < 16 || K > HEAD_MAX_K || K % 16 != 0)
        return fail(SPIKE_EINVAL, "K = %d must be a multiple of 16 in [16, %d]", K, HEAD_MAX_K);
    if (V < 1 || (int64_t)V * K >= ((int64_t)1 << 31))
        return fail(SPIKE_EINVAL, "V = %d outside [1, 2^31 / K)", V);
    if (top_k < 1 || top_k > HEAD_MAX_TOP_K || top_k > V)
        return fail(SPIKE_EINVAL, "top_k = %d outside [1, min(%d, V = %d)]", top_k, HEAD_MAX_TOP_K, V);
    if (std::isnan(threshold))
        return fail(SPIKE_EINVAL, "threshold is NaN");
    if (!Q || !scale || !x || !logits || !cand || !cand_logits || !result || !workspace)
        return fail(SPIKE_EINVAL, "null pointer argument");
    if (!aligned(Q, 16) || !aligned(workspace, 16))
        return fail(SPIKE_EINVAL, "Q and the workspace must be 16-byte aligned");
    if (!aligned(scale, 4) || !aligned(x, 4) || !aligned(logits, 4) || !aligned(cand, 4) ||
        !aligned(cand_logits, 4) || !aligned(result, 4))
        return fail(SPIKE_EINVAL, "scale, x and the outputs must be 4-byte aligned");
    const hipStream_t st = static_cast<hipStream_t>(stream);
    auto* ws = static_cast<spk::HeadWorkspace*>(workspace);
    const int npl = (K + 511) / 512;
    const int64_t groups = ((int64_t)V + 1) / 2 * 2;
    const int64_t wgs = std::max<int64_t>(1, std::min<int64_t>((groups + spk::kRegGroups - 1) / spk::kRegGroups,
                                                               spk::kApproxMaxWgs));
    // a gap is never negative, so only a threshold > 0 can ask for verification:
    // then the approximate head also computes every row's FP32-activation logit
    const bool spec = threshold > 0.0f;
    // with the FP32 activations also in registers, K > 2048 leaves room for
    // one wave per SIMD: the grid is then what fits at once (results do not
    // depend on the grid)
    const int64_t grid = spec && npl > 4 ? std::min<int64_t>(wgs, 256) : wgs;
    hipLaunchKernelGGL(spec ? pick_approx<true>(npl) : pick_approx<false>(npl), dim3((unsigned)grid),
                       dim3(spk::kRegBlock), 0, st, Q, scale, K, V, x, logits, ws);
    hipLaunchKernelGGL(spk::k_head_select, dim3(1), dim3(spk::kSelectBlock), 0, st, logits, V, top_k, threshold,
                       (int)grid, (int)spec, ws, Q, scale, K, x, cand, cand_logits, result);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "head verification launch");
    return SPIKE_OK;
}

}  // extern "C"
