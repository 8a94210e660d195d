// Pooling layers of the networks the shift operators run in (the ResNet-18 of
// the paper's Section 6 timing has a 3 x 3 stride-2 max pool after its stem and
// a global average pool before its classifier), on int32 fixed point.
// Both are small, memory-bound passes: one thread per output.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "common.hpp"

namespace ds {

namespace {

// One thread per output; the window positions in the padding are skipped.
__global__ void __launch_bounds__(256)
maxpool_kernel(const int32_t *__restrict__ x, int32_t *__restrict__ y, int64_t total, int H, int W,
               int OH, int OW, int R, int S, int sh, int sw, int ph, int pw)
{
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int ow = int(idx % OW);
        int64_t t = idx / OW;
        const int oh = int(t % OH);
        const int64_t plane = t / OH;  // n * C + c
        const int32_t *xp = x + plane * H * W;
        int32_t best = INT_MIN;
        for (int r = 0; r < R; ++r) {
            const int ih = oh * sh - ph + r;
            if (ih < 0 || ih >= H) continue;
            for (int s = 0; s < S; ++s) {
                const int iw = ow * sw - pw + s;
                if (iw < 0 || iw >= W) continue;
                best = max(best, xp[ih * W + iw]);
            }
        }
        y[idx] = best;
    }
}

// One thread per (n, c) plane: floor of the int64 sum over the plane / HW.
__global__ void __launch_bounds__(256)
avgpool_global_kernel(const int32_t *__restrict__ x, int32_t *__restrict__ y, int64_t planes,
                      int HW)
{
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < planes;
         i += int64_t(gridDim.x) * blockDim.x) {
        const int32_t *xp = x + i * HW;
        int64_t sum = 0;
        for (int p = 0; p < HW; ++p) sum += xp[p];
        int64_t q = sum / HW;
        if (sum % HW != 0 && sum < 0) q -= 1;  // division truncates; floor it
        y[i] = int32_t(q);
    }
}

ds_status status_of(hipError_t e, const char *what)
{
    if (e == hipSuccess) return ok();
    return fail(DS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int grid_for(int64_t total)
{
    return int(std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 8192)));
}

}  // namespace

}  // namespace ds

using namespace ds;

extern "C" ds_status ds_maxpool2d(const int32_t *x, int32_t *y, int64_t n, int64_t c, int64_t h,
                                  int64_t w, int64_t r, int64_t s, int32_t stride_h,
                                  int32_t stride_w, int32_t pad_h, int32_t pad_w, uint32_t flags,
                                  void *stream)
{
    if (!x || !y) return fail(DS_ERR_NULL_POINTER, "x and y must not be NULL");
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0 || r <= 0 || s <= 0)
        return fail(DS_ERR_INVALID_SHAPE, "all sizes must be > 0");
    if (stride_h < 1 || stride_w < 1) return fail(DS_ERR_INVALID_ARG, "stride must be >= 1");
    if (pad_h < 0 || pad_w < 0 || 2 * int64_t(pad_h) > r || 2 * int64_t(pad_w) > s)
        return fail(DS_ERR_INVALID_ARG, "padding must be in [0, kernel / 2]");
    if (h + 2 * int64_t(pad_h) < r || w + 2 * int64_t(pad_w) < s)
        return fail(DS_ERR_INVALID_SHAPE, "window larger than the padded input");
    if (flags != 0) return fail(DS_ERR_INVALID_ARG, "flags must be 0");
    const int64_t oh = (h + 2 * int64_t(pad_h) - r) / stride_h + 1;
    const int64_t ow = (w + 2 * int64_t(pad_w) - s) / stride_w + 1;
    const int64_t xe = prod({n, c, h, w}), ye = prod({n, c, oh, ow});
    if (xe < 0 || ye < 0 || xe > kMaxElems || ye > kMaxElems || r > kMaxElems || s > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    if (overlap(x, 4 * xe, y, 4 * ye)) return fail(DS_ERR_INVALID_ARG, "y overlaps x");
    if (!device_range_ok(x, 4 * xe)) return fail(DS_ERR_INVALID_ARG, "x is not a device buffer of %lld bytes", (long long)(4 * xe));
    if (!device_range_ok(y, 4 * ye)) return fail(DS_ERR_INVALID_ARG, "y is not a device buffer of %lld bytes", (long long)(4 * ye));
    hipLaunchKernelGGL(maxpool_kernel, dim3(grid_for(ye)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), x, y, ye, int(h), int(w), int(oh),
                       int(ow), int(r), int(s), stride_h, stride_w, pad_h, pad_w);
    return status_of(hipGetLastError(), "ds_maxpool2d");
}

extern "C" ds_status ds_avgpool2d_global(const int32_t *x, int32_t *y, int64_t n, int64_t c,
                                         int64_t h, int64_t w, uint32_t flags, void *stream)
{
    if (!x || !y) return fail(DS_ERR_NULL_POINTER, "x and y must not be NULL");
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0) return fail(DS_ERR_INVALID_SHAPE, "all sizes must be > 0");
    if (flags != 0) return fail(DS_ERR_INVALID_ARG, "flags must be 0");
    const int64_t xe = prod({n, c, h, w}), ye = prod({n, c});
    if (xe < 0 || xe > kMaxElems) return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    if (overlap(x, 4 * xe, y, 4 * ye)) return fail(DS_ERR_INVALID_ARG, "y overlaps x");
    if (!device_range_ok(x, 4 * xe)) return fail(DS_ERR_INVALID_ARG, "x is not a device buffer of %lld bytes", (long long)(4 * xe));
    if (!device_range_ok(y, 4 * ye)) return fail(DS_ERR_INVALID_ARG, "y is not a device buffer of %lld bytes", (long long)(4 * ye));
    hipLaunchKernelGGL(avgpool_global_kernel, dim3(grid_for(ye)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), x, y, ye, int(h * w));
    return status_of(hipGetLastError(), "ds_avgpool2d_global");
}
