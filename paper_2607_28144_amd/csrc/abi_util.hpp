// Status and error-text helpers of the C ABI, shared by the entry-point
// files (defined in api.cpp, which keeps the thread-local error text).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>

#include "regenvc_attn.h"

namespace regenvc {
namespace abi {

// Records msg as this thread's last error and returns st.
regenvc_status fail_msg(regenvc_status st, const char *msg);
// REGENVC_OK if the current device is gfx950 (cached per device).
regenvc_status device_ok();
// REGENVC_ERR_HIP with the runtime's text if e is an error, else REGENVC_OK
// (clearing the last error).
regenvc_status launch_status(hipError_t e, const char *what);
void clear_error();

inline regenvc_status failf(regenvc_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    return fail_msg(st, buf);
}

// Byte range [lo, hi) of a buffer, for overlap checks.
struct Range {
    uintptr_t lo, hi;
};
inline Range range_of(const void *p, int64_t bytes)
{
    const uintptr_t b = reinterpret_cast<uintptr_t>(p);
    return Range{b, b + (uintptr_t)bytes};
}
inline bool overlaps(const Range &a, const Range &b)
{
    return a.lo < b.hi && b.lo < a.hi;
}
inline bool aligned(const void *p, unsigned n)
{
    return reinterpret_cast<uintptr_t>(p) % n == 0;
}

}  // namespace abi
}  // namespace regenvc
