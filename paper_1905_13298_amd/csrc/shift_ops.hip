// Entry points of the shift operators (DeepShift Section 3, LinearShift and
// ConvShift) and their argument checks. LinearShift runs as a ConvShift with
// H = W = R = S = 1: x [batch][in] is x [n][c][1][1] and y [batch][out] is
// y [n][k][1][1], so both operators share every kernel.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.hpp"
#include "conv_plan.hpp"

namespace ds {

bool device_range_ok(const void *p, int64_t bytes)
{
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void *>(p)) != hipSuccess) {
        (void)hipGetLastError();  // clear the sticky error of a failed lookup
        return false;
    }
    auto b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
    return q >= b && q - b + uint64_t(bytes) <= uint64_t(size);
}

// Validates the sizes of a convolution problem and fills `g` (no pointers).
static ds_status check_shape(int64_t n, int64_t c, int64_t h, int64_t w, int64_t k, int64_t r,
                             int64_t s, int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                             bool packed, ConvGeom &g, int bits = 5)
{
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0 || k <= 0 || r <= 0 || s <= 0)
        return fail(DS_ERR_INVALID_SHAPE, "all sizes must be > 0");
    if (sh < 1 || sw < 1) return fail(DS_ERR_INVALID_ARG, "stride must be >= 1");
    if (ph < 0 || pw < 0) return fail(DS_ERR_INVALID_ARG, "padding must be >= 0");
    if (h + 2 * int64_t(ph) < r || w + 2 * int64_t(pw) < s)
        return fail(DS_ERR_INVALID_SHAPE, "kernel larger than the padded input");
    const int64_t oh = (h + 2 * int64_t(ph) - r) / sh + 1;
    const int64_t ow = (w + 2 * int64_t(pw) - s) / sw + 1;
    const int64_t crs = prod({c, r, s});
    const int64_t xe = prod({n, c, h, w}), ye = prod({n, k, oh, ow});
    const int64_t we = packed ? prod({k, row_words_bits(crs, bits)}) : prod({k, crs});
    if (crs < 0 || xe < 0 || ye < 0 || we < 0 || crs > kMaxElems || xe > kMaxElems ||
        ye > kMaxElems || we > kMaxElems || prod({k, crs}) > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    g = ConvGeom{int(n), int(c), int(h), int(w), int(k), int(r), int(s), sh, sw, ph, pw,
                 int(oh), int(ow), int(crs), bits};
    return DS_SUCCESS;
}

// Validates a convolution problem (both operators) and fills `g`.
static ds_status check_conv(const void *x, const void *wts, const void *bias, const void *y,
                            int64_t n, int64_t c, int64_t h, int64_t w, int64_t k, int64_t r,
                            int64_t s, int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                            int32_t frac_bits, uint32_t flags, bool packed, ConvGeom &g,
                            uint32_t allowed_flags)
{
    if (!x || !wts || !y) return fail(DS_ERR_NULL_POINTER, "x, weights and y must not be NULL");
    if (packed) allowed_flags |= 0xF00u;                 // DS_CODE_BITS field
    const int bits = packed ? flags_code_bits(flags) : 5;
    ds_status st = check_shape(n, c, h, w, k, r, s, sh, sw, ph, pw, packed, g, bits < 0 ? 5 : bits);
    if (st != DS_SUCCESS) return st;
    if (frac_bits < 0 || frac_bits > 31) return fail(DS_ERR_INVALID_ARG, "frac_bits must be in [0, 31]");
    if (flags & ~allowed_flags) return fail(DS_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
    if (bits < 0) return fail(DS_ERR_INVALID_ARG, "DS_CODE_BITS must be 2..5 (or 0 for 5)");
    const int64_t xb = 4 * int64_t(g.n) * g.c * g.h * g.w;
    const int64_t yb = 4 * int64_t(g.n) * g.k * g.oh * g.ow;
    const int64_t wb = 4 * (packed ? int64_t(g.k) * row_words_bits(g.crs, g.bits) : int64_t(g.k) * g.crs);
    const int64_t bb = 4 * int64_t(g.k);
    if (overlap(y, yb, x, xb) || overlap(y, yb, wts, wb) || overlap(y, yb, bias, bb))
        return fail(DS_ERR_INVALID_ARG, "y overlaps an input");
    if (!device_range_ok(x, xb)) return fail(DS_ERR_INVALID_ARG, "x is not a device buffer of %lld bytes", (long long)xb);
    if (!device_range_ok(wts, wb)) return fail(DS_ERR_INVALID_ARG, "weights are not a device buffer of %lld bytes", (long long)wb);
    if (!device_range_ok(y, yb)) return fail(DS_ERR_INVALID_ARG, "y is not a device buffer of %lld bytes", (long long)yb);
    if (bias && !device_range_ok(bias, bb)) return fail(DS_ERR_INVALID_ARG, "bias is not a device buffer of %lld bytes", (long long)bb);
    return DS_SUCCESS;
}

static ds_status hip_status(hipError_t e, const char *what)
{
    if (e == hipSuccess) return ok();
    return fail(DS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace ds

using namespace ds;

extern "C" ds_status ds_conv2d_shift(const int32_t *x, const uint32_t *w_packed, const int32_t *bias,
                                     int32_t *y, int64_t n, int64_t c, int64_t h, int64_t w,
                                     int64_t k, int64_t r, int64_t s, int32_t stride_h,
                                     int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                     int32_t frac_bits, uint32_t flags, void *stream)
{
    ConvGeom g;
    ds_status st = check_conv(x, w_packed, bias, y, n, c, h, w, k, r, s, stride_h, stride_w,
                              pad_h, pad_w, frac_bits, flags, true, g, DS_RELU);
    if (st != DS_SUCCESS) return st;
    Epilogue epi;
    epi.relu = (flags & DS_RELU) != 0;
    return hip_status(run_conv(g, x, w_packed, nullptr, bias, y, Inner::Shift,
                               static_cast<hipStream_t>(stream), epi),
                      "ds_conv2d_shift");
}

extern "C" ds_status ds_conv2d_shift_fused(const int32_t *x, const uint32_t *w_packed,
                                           const int32_t *bias, const int32_t *mul,
                                           const int32_t *add, int32_t mul_shift,
                                           const int32_t *residual, int32_t *y, int64_t n,
                                           int64_t c, int64_t h, int64_t w, int64_t k, int64_t r,
                                           int64_t s, int32_t stride_h, int32_t stride_w,
                                           int32_t pad_h, int32_t pad_w, int32_t frac_bits,
                                           uint32_t flags, void *stream)
{
    ConvGeom g;
    // Arguments first (no device access), then the buffers.
    if (x && w_packed && y) {
        const int bits = flags_code_bits(flags);
        ds_status st = check_shape(n, c, h, w, k, r, s, stride_h, stride_w, pad_h, pad_w, true, g,
                                   bits < 0 ? 5 : bits);
        if (st != DS_SUCCESS) return st;
        if (add && !mul) return fail(DS_ERR_INVALID_ARG, "add needs mul");
        if (mul_shift < 0 || mul_shift > 31) return fail(DS_ERR_INVALID_ARG, "mul_shift must be in [0, 31]");
        const int64_t kb = 4 * int64_t(g.k);
        const int64_t yb = 4 * int64_t(g.n) * g.k * g.oh * g.ow;
        if (overlap(y, yb, mul, kb) || overlap(y, yb, add, kb) || overlap(y, yb, residual, yb))
            return fail(DS_ERR_INVALID_ARG, "y overlaps an input");
    }
    ds_status st = check_conv(x, w_packed, bias, y, n, c, h, w, k, r, s, stride_h, stride_w,
                              pad_h, pad_w, frac_bits, flags, true, g, DS_RELU);
    if (st != DS_SUCCESS) return st;
    const int64_t kb = 4 * int64_t(g.k);
    const int64_t yb = 4 * int64_t(g.n) * g.k * g.oh * g.ow;
    if (mul && !device_range_ok(mul, kb)) return fail(DS_ERR_INVALID_ARG, "mul is not a device buffer of %lld bytes", (long long)kb);
    if (add && !device_range_ok(add, kb)) return fail(DS_ERR_INVALID_ARG, "add is not a device buffer of %lld bytes", (long long)kb);
    if (residual && !device_range_ok(residual, yb))
        return fail(DS_ERR_INVALID_ARG, "residual is not a device buffer of %lld bytes", (long long)yb);
    Epilogue epi;
    epi.mul = mul;
    epi.add = add;
    epi.mul_shift = mul_shift;
    epi.res = residual;
    epi.relu = (flags & DS_RELU) != 0;
    return hip_status(run_conv(g, x, w_packed, nullptr, bias, y, Inner::Shift,
                               static_cast<hipStream_t>(stream), epi),
                      "ds_conv2d_shift_fused");
}

extern "C" ds_status ds_linear_shift(const int32_t *x, const uint32_t *w_packed, const int32_t *bias,
                                     int32_t *y, int64_t batch, int64_t in_features,
                                     int64_t out_features, int32_t frac_bits, uint32_t flags,
                                     void *stream)
{
    ConvGeom g;
    ds_status st = check_conv(x, w_packed, bias, y, batch, in_features, 1, 1, out_features, 1, 1,
                              1, 1, 0, 0, frac_bits, flags, true, g, DS_RELU);
    if (st != DS_SUCCESS) return st;
    Epilogue epi;
    epi.relu = (flags & DS_RELU) != 0;
    return hip_status(run_conv(g, x, w_packed, nullptr, bias, y, Inner::Shift,
                               static_cast<hipStream_t>(stream), epi),
                      "ds_linear_shift");
}

extern "C" ds_status ds_conv2d_shift_describe(int64_t n, int64_t c, int64_t h, int64_t w,
                                              int64_t k, int64_t r, int64_t s, int32_t stride_h,
                                              int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                              char *buf, int64_t len)
{
    if (!buf) return fail(DS_ERR_NULL_POINTER, "buf must not be NULL");
    if (len < 1) return fail(DS_ERR_BUFFER_TOO_SMALL, "len must be >= 1");
    ConvGeom g;
    const ds_status st = check_shape(n, c, h, w, k, r, s, stride_h, stride_w, pad_h, pad_w, true, g);
    if (st != DS_SUCCESS) return st;
    describe_conv(g, buf, size_t(len));
    return ok();
}

extern "C" ds_status ds_conv2d_mul_i32(const int32_t *x, const int32_t *wts, const int32_t *bias,
                                       int32_t *y, int64_t n, int64_t c, int64_t h, int64_t w,
                                       int64_t k, int64_t r, int64_t s, int32_t stride_h,
                                       int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                       uint32_t flags, void *stream)
{
    ConvGeom g;
    ds_status st = check_conv(x, wts, bias, y, n, c, h, w, k, r, s, stride_h, stride_w, pad_h,
                              pad_w, 0, flags, false, g, DS_MUL_I24);
    if (st != DS_SUCCESS) return st;
    return hip_status(run_conv(g, x, nullptr, wts, bias, y, (flags & DS_MUL_I24) ? Inner::Mul24 : Inner::Mul,
                               static_cast<hipStream_t>(stream)),
                      "ds_conv2d_mul_i32");
}

extern "C" ds_status ds_linear_mul_i32(const int32_t *x, const int32_t *wts, const int32_t *bias,
                                       int32_t *y, int64_t batch, int64_t in_features,
                                       int64_t out_features, uint32_t flags, void *stream)
{
    ConvGeom g;
    ds_status st = check_conv(x, wts, bias, y, batch, in_features, 1, 1, out_features, 1, 1, 1,
                              1, 0, 0, 0, flags, false, g, DS_MUL_I24);
    if (st != DS_SUCCESS) return st;
    return hip_status(run_conv(g, x, nullptr, wts, bias, y, (flags & DS_MUL_I24) ? Inner::Mul24 : Inner::Mul,
                               static_cast<hipStream_t>(stream)),
                      "ds_linear_mul_i32");
}

// ---------------------------------------------------------------------------
// ConvShift without allocation. The scratch of the runtime kernel (decoded
// weights, per-channel start values, transposed operands of a LinearShift)
// lives in this array, one copy per GPU in the library's code object, held
// from the code object's load on that GPU to the end of the process. The
// array's name is a host-side stand-in: host code takes the device address of
// the current GPU's copy from hipGetSymbolAddress, once per device, and passes
// that address on.

static __device__ __align__(256) unsigned char scratch[DS_NOALLOC_SCRATCH_BYTES];

namespace ds {
namespace {

constexpr int kMaxDevices = 64;

// Device address of the current device's copy of `scratch`, looked up on the
// first call on that device (with the device current).
hipError_t noalloc_scratch(void **out)
{
    static std::mutex mu;
    static void *ptr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        ptr[dev] = p;
    }
    *out = ptr[dev];
    return hipSuccess;
}

}  // namespace
}  // namespace ds

extern "C" ds_status ds_conv2d_shift_noalloc(const int32_t *x, const uint32_t *w_packed,
                                             const int32_t *bias, int32_t *y, int64_t n, int64_t c,
                                             int64_t h, int64_t w, int64_t k, int64_t r, int64_t s,
                                             int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                             int32_t pad_w, int32_t frac_bits, uint32_t flags,
                                             void *stream)
{
    ConvGeom g;
    // The size limit is checked from the shape alone, before any device access.
    if (x && w_packed && y) {
        const int bits = flags_code_bits(flags);
        ds_status st = check_shape(n, c, h, w, k, r, s, stride_h, stride_w, pad_h, pad_w, true, g,
                                   bits < 0 ? 5 : bits);
        if (st != DS_SUCCESS) return st;
        const size_t need = conv_scratch_bytes(g);
        if (need > size_t(DS_NOALLOC_SCRATCH_BYTES))
            return fail(DS_ERR_UNSUPPORTED,
                        "ds_conv2d_shift_noalloc: this problem needs %zu bytes of scratch, more than "
                        "the %u bytes the library holds for it (use ds_conv2d_shift)",
                        need, unsigned(DS_NOALLOC_SCRATCH_BYTES));
    }
    ds_status st = check_conv(x, w_packed, bias, y, n, c, h, w, k, r, s, stride_h, stride_w,
                              pad_h, pad_w, frac_bits, flags, true, g, DS_RELU);
    if (st != DS_SUCCESS) return st;
    void *ws = nullptr;
    const hipError_t e = noalloc_scratch(&ws);
    if (e != hipSuccess) return hip_status(e, "ds_conv2d_shift_noalloc: scratch address");
    Epilogue epi;
    epi.relu = (flags & DS_RELU) != 0;
    return hip_status(run_conv(g, x, w_packed, nullptr, bias, y, Inner::Shift,
                               static_cast<hipStream_t>(stream), epi, OutMap(), Padded(),
                               Workspace{ws, size_t(DS_NOALLOC_SCRATCH_BYTES)}),
                      "ds_conv2d_shift_noalloc");
}

extern "C" int64_t ds_conv2d_shift_noalloc_scratch_bytes(int64_t n, int64_t c, int64_t h, int64_t w,
                                                         int64_t k, int64_t r, int64_t s,
                                                         int32_t stride_h, int32_t stride_w,
                                                         int32_t pad_h, int32_t pad_w)
{
    ConvGeom g;
    if (check_shape(n, c, h, w, k, r, s, stride_h, stride_w, pad_h, pad_w, true, g) != DS_SUCCESS)
        return -1;
    ok();
    return int64_t(conv_scratch_bytes(g));
}
