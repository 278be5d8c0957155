// Internal helpers of the APEX library: error reporting and argument checks.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "apex.h"

namespace apex {

// Records the message for apex_last_error() on the calling thread and returns `st`.
apex_status fail(apex_status st, const char *fmt, ...);

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace apex

#define APEX_REQUIRE(cond, ...)                                  \
    do {                                                         \
        if (!(cond)) return ::apex::fail(APEX_E_INVAL, __VA_ARGS__); \
    } while (0)

#define APEX_HIP(call)                                                          \
    do {                                                                        \
        hipError_t apex_err_ = (call);                                          \
        if (apex_err_ != hipSuccess)                                            \
            return ::apex::fail(APEX_E_HIP, "%s failed: %s", #call,            \
                                hipGetErrorString(apex_err_));                  \
    } while (0)
