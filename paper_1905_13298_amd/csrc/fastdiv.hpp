// Division by a launch-constant divisor for dividends below 2^31
// (round-up multiplier method of Granlund and Montgomery, 1994): the host
// computes the multiplier once, the kernel divides with one multiply-high,
// an add and a shift.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ds {

struct FastDiv {
    uint32_t d, m, l;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{d, uint32_t(m), l};
}

__device__ __forceinline__ int fdiv(int n, const FastDiv &f)
{
    return int((__umulhi(uint32_t(n), f.m) + uint32_t(n)) >> f.l);
}

}  // namespace ds
