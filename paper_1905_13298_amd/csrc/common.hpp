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

// Words of a packed row of `cols` codes of `bits` bits (floor(32 / bits) per word).
inline int64_t row_words_bits(int64_t cols, int bits)
{
    const int per = 32 / bits;
    return cols <= 0 ? -1 : (cols + per - 1) / per;
}

#if defined(__HIPCC__)
#define DS_HD __host__ __device__
#else
#define DS_HD
#endif

// Packed weight codes of `bits` bits (2..5): floor(32 / bits) codes per uint32
// word, code j of a word in bits [bits*j, bits*j + bits). The top bit of a code
// is the sign, the others the shift code, all ones meaning a zero weight; for
// 5 bits this is the canonical code (bit 4 sign, shift code 15 = zero).
// Shared by the host packer and the device kernels.
struct CodeFmt {
    int bits = 5, per_word = 6;
    // The canonical 5-bit code of a raw `bits`-bit code.
    DS_HD uint32_t canonical(uint32_t raw) const
    {
        const uint32_t shmask = (1u << (bits - 1)) - 1u;
        const uint32_t sh = raw & shmask, sign = (raw >> (bits - 1)) & 1u;
        return (sign << 4) | (sh == shmask ? 15u : sh);
    }
    // Canonical code j of a packed row (j < 2^31). The 5-bit format, the common
    // one, divides by a constant.
    DS_HD uint32_t at(const uint32_t *row, int j) const
    {
        const int q = bits == 5 ? j / 6 : j / per_word;
        const uint32_t word = row[q];
        return canonical((word >> (bits * (j - q * per_word))) & ((1u << bits) - 1u));
    }
};

inline CodeFmt code_fmt(int bits) { return CodeFmt{bits, 32 / bits}; }

// Code width carried in bits 8-11 of a flags word (DS_CODE_BITS); 0 means 5.
// Returns -1 for a width outside 2..5.
inline int flags_code_bits(uint32_t flags)
{
    const int b = int((flags >> 8) & 15u);
    if (b == 0) return 5;
    return b >= 2 && b <= 5 ? b : -1;
}

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
