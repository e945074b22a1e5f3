// Error reporting shared by the library's entry points: the calling
// thread's last failure message (spike_proj_last_error) and the code.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "spike_proj.h"

namespace spk {

inline thread_local std::string last_error;

inline int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    last_error = buf;
    return code;
}

inline int hip_fail(hipError_t e, const char* what)
{
    return fail(SPIKE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace spk
