// Problem geometry and the launch entry shared by the operator front ends.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ds {

// One convolution problem (LinearShift is the case h = w = r = s = 1).
struct ConvGeom {
    int n, c, h, w, k, r, s;
    int sh, sw, ph, pw;
    int oh, ow;
    int crs;
};

// Inner operation of the reduction: the DeepShift shift-accumulate, or the
// multiplication-based comparison (int32 multiply-add).
enum class Inner { Shift, Mul };

// Enqueue the whole computation of y on `stream`. Exactly one of `wpacked`
// (Shift) and `wint` (Mul) is used.
hipError_t run_conv(const ConvGeom &g, const int32_t *x, const uint32_t *wpacked,
                    const int32_t *wint, const int32_t *bias, int32_t *y, Inner op,
                    hipStream_t stream);

// Kernel variant forced for testing: -1 = automatic choice, 0 = the
// one-thread-per-output kernel, 1 = the tiled kernel. Set from the environment
// variable DS_FORCE_VARIANT when the library loads.
int forced_variant();

}  // namespace ds
