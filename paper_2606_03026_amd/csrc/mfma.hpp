// Dense i8 matrix-core contraction over the 0/1 spike matrix (prefill-sized
// batches).  Placeholder until the kernel lands: reports itself unsupported,
// so AUTO dispatch keeps every batch on the gather path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spk {

constexpr int kMfmaNAlign = 64;

inline bool mfma_supported(int K, int N, const void* W)
{
    (void)K;
    (void)N;
    (void)W;
    return false;
}

inline hipError_t launch_mfma(const int8_t*, const float*, int, int, const uint64_t*, int, float*, int32_t*, bool,
                              hipStream_t)
{
    return hipErrorNotSupported;
}

}  // namespace spk
