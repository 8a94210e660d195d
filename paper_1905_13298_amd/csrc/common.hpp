// Host-side helpers shared by the entry points: error reporting and argument
// validation. Nothing here touches the device except device_range_ok().
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "deepshift.h"

namespace ds {

// Per-thread detail for the last error (returned by ds_last_error_message).
std::string &last_error();

inline ds_status fail(ds_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    last_error() = buf;
    return st;
}

inline ds_status ok()
{
    last_error().clear();
    return DS_SUCCESS;
}

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;  // per tensor

inline int64_t row_words(int64_t cols) { return cols <= 0 ? -1 : (cols + 5) / 6; }

// Overflow-safe product of positive sizes; returns -1 when it exceeds 2^62.
inline int64_t prod(std::initializer_list<int64_t> v)
{
    int64_t p = 1;
    for (int64_t a : v) {
        if (a <= 0) return 0;
        if (p > (int64_t(1) << 62) / a) return -1;
        p *= a;
    }
    return p;
}

inline bool overlap(const void *a, int64_t abytes, const void *b, int64_t bbytes)
{
    if (!a || !b) return false;
    auto a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + uintptr_t(bbytes) && b0 < a0 + uintptr_t(abytes);
}

// True when [p, p + bytes) lies inside one device allocation known to the HIP
// runtime. Rejects host pointers and buffers too small for the shape.
bool device_range_ok(const void *p, int64_t bytes);

}  // namespace ds
