// Thread-local error messages behind slw_last_error().
#include <cstdarg>
#include <cstdio>

#include "common.h"

namespace {
thread_local char g_msg[512] = "";
}

namespace slw {

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_msg[0] = '\0'; }

}  // namespace slw

extern "C" const char* slw_last_error(void) { return g_msg; }
