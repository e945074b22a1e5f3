// Vector types and buffer-resource helpers shared by the kernels (gfx950).
//
// A buffer resource holds a base address and a size in scalar registers;
// each lane supplies a 32-bit byte offset.  There is no 64-bit address
// arithmetic per lane, and an offset at or past the resource's size reads
// as zero without a memory access, so the kernels load unconditionally and
// point lanes with nothing to read at kOutOfRange.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spk {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kOutOfRange = 0x80000000u;  // offset that is always past the resource
constexpr int64_t kBufMaxBytes = 0x7fffff00;   // largest matrix one resource addresses
constexpr int kBufferFlags = 0x00020000;       // buffer resource word 3: 32-bit data format (gfx9)

__device__ inline __amdgpu_buffer_rsrc_t weight_resource(const int8_t* base, int64_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(base), 0, (int)bytes, kBufferFlags);
}

}  // namespace spk
