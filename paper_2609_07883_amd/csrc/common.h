// Internal helpers shared by the host-side translation units of libsloweave.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "sloweave.h"

namespace slw {

// Records a thread-local message for slw_last_error() and returns `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Wraps a body so that no C++ exception crosses the C ABI.
template <class F>
int guarded(F&& f) {
    try {
        return f();
    } catch (const std::bad_alloc&) {
        return fail(SLW_ENOMEM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(SLW_EINVAL, "internal error: %s", e.what());
    } catch (...) {
        return fail(SLW_EINVAL, "internal error");
    }
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace slw
