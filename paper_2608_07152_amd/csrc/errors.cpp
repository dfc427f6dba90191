// Thread-local last-error message of libeahr, and the trace switch.
#include <cstdarg>
#include <cstdio>
#include <cstdlib>

#include "common.h"

namespace {
thread_local char g_err[512] = "";
}

namespace eahr {
void set_error(const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
}

bool trace_on() {
    static const bool on = [] {
        const char* p = std::getenv("EAHR_TRACE");
        return p && *p && *p != '0';
    }();
    return on;
}
}  // namespace eahr

extern "C" const char* eahr_last_error(void) { return g_err; }
