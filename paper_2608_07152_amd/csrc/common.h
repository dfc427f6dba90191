// Error reporting shared by the host parts of libeahr.
#pragma once
#include <cstdarg>
#include <cstdio>

#include "eahr.h"

namespace eahr {
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));

// EAHR_TRACE=1 (environment) turns on per-round timing lines on stderr: one
// per depth round of eahr_topk and one per scan round of the dense channel.
bool trace_on();
}

#define EAHR_FAIL(code, ...)           \
    do {                               \
        ::eahr::set_error(__VA_ARGS__); \
        return (code);                 \
    } while (0)

#define HIP_TRY(expr)                                                               \
    do {                                                                            \
        hipError_t e_ = (expr);                                                     \
        if (e_ != hipSuccess) {                                                     \
            ::eahr::set_error("%s failed: %s", #expr, hipGetErrorString(e_));       \
            return (e_ == hipErrorOutOfMemory) ? EAHR_E_OOM : EAHR_E_HIP;           \
        }                                                                           \
    } while (0)

#define EAHR_TRY(expr)          \
    do {                        \
        int rc_ = (expr);       \
        if (rc_ != EAHR_OK) return rc_; \
    } while (0)
