// Thread-local error message and ABI version.
#include <cstdarg>
#include <cstdio>

#include "common.h"

namespace {
thread_local char g_last_error[512] = "";
}

namespace apex {
apex_status fail(apex_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}
}  // namespace apex

extern "C" int apex_abi_version(void) { return APEX_ABI_VERSION; }
extern "C" const char *apex_last_error(void) { return g_last_error; }
