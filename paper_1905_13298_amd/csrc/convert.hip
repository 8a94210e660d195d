// Float -> shift-code converter and float -> fixed-point conversion, the steps
// that feed the shift operators:
//   * DeepShift-Q (Section 3, Eqs. 4-5): sign(w) and round(log2|w|);
//   * DeepShift-PS (Section 3): round(P) and the ternary sign thresholds +-0.5;
//   * the power is clipped to -max_shift .. 0 (Section 4, 14 for 5-bit codes);
//   * inputs and bias rounded to fixed point with F fractional bits
//     (Section 4, 16.16).
// The weight converters write the packed 5-bit format directly.
//
// Both are streaming kernels bound by HBM bandwidth. A weight block owns 256
// consecutive packed words. The floats those words cover form one contiguous
// range (rows are stored back to back), so the block reads that range with
// coalesced loads, turns every float into its code once, keeps the codes as
// bytes in LDS, and then each thread gathers the six codes of its word and
// stores the word (coalesced).
#include <hip/hip_runtime.h>

#include <cmath>

#include "common.hpp"

namespace ds {

namespace {

constexpr int kWordsPerBlock = 256;
constexpr int kCodesPerWord = 6;
constexpr uint32_t kZeroCode = 15;

// Code of flip(2^p, s) for p already clipped to -max_shift .. 0.
__device__ __forceinline__ uint32_t make_code(int p, bool negative)
{
    return (negative ? 16u : 0u) | uint32_t(-p);
}

// DeepShift-Q code of one float, from its bits. For a normal float
// |w| = 1.m * 2^e, floor(log2|w|) = e and round(log2|w|) = e + 1 exactly when
// 1.m >= sqrt(2), i.e. when the 23-bit mantissa field is at least
// ceil((sqrt(2) - 1) * 2^23) = 0x3504F4 (sqrt(2) * 2^23 = 11863283.2...).
// Subnormals lie below 2^-126 and clip to -max_shift; +-inf clip to 0.
__device__ __forceinline__ uint32_t code_q(float w, int max_shift)
{
    const uint32_t b = __float_as_uint(w);
    const uint32_t mag = b & 0x7fffffffu;
    if (mag == 0 || mag > 0x7f800000u) return kZeroCode;  // +-0 and NaN: sign 0
    const int e = int(mag >> 23);
    int p;
    if (e == 0) {
        p = -max_shift;                                   // subnormal
    } else {
        p = e - 127 + ((mag & 0x7fffffu) >= 0x3504f4u ? 1 : 0);  // inf: e = 255 -> > 0
        p = p > 0 ? 0 : (p < -max_shift ? -max_shift : p);
    }
    return make_code(p, (b >> 31) != 0);
}

// DeepShift-PS code from one shift parameter and one sign parameter. roundf
// rounds halves away from zero, the tie rule the sign thresholds imply.
__device__ __forceinline__ uint32_t code_ps(float pv, float sv, int max_shift)
{
    const bool neg = sv <= -0.5f, pos = sv >= 0.5f;       // NaN: neither
    const float r = roundf(pv);
    if (!(neg || pos) || r != r) return kZeroCode;
    const float c = fminf(fmaxf(r, float(-max_shift)), 0.0f);
    return make_code(int(c), neg);
}

struct WordRange {
    int64_t first_float;  // flat index of the first float of word t
    int ncodes;           // codes of word t that come from the row (1..6)
};

__device__ __forceinline__ WordRange word_range(int64_t t, int64_t cols, int64_t wpr)
{
    const int64_t row = t / wpr, j = t - row * wpr;
    const int64_t col = j * kCodesPerWord;
    WordRange r;
    r.first_float = row * cols + col;
    r.ncodes = int(min<int64_t>(kCodesPerWord, cols - col));
    return r;
}

template <bool PS>
__global__ __launch_bounds__(kWordsPerBlock) void quantize_kernel(
    const float *__restrict__ w, const float *__restrict__ sgn, int64_t cols, int64_t wpr,
    int64_t nwords, int max_shift, uint32_t *__restrict__ out)
{
    __shared__ uint8_t codes[kWordsPerBlock * kCodesPerWord];
    const int64_t t0 = int64_t(blockIdx.x) * kWordsPerBlock;
    const int64_t t1 = min<int64_t>(t0 + kWordsPerBlock, nwords);
    // Floats covered by words [t0, t1): [f0, f1). Word t1 (or the end) starts at f1.
    const int64_t f0 = word_range(t0, cols, wpr).first_float;
    const int64_t f1 = t1 == nwords ? (nwords / wpr) * cols : word_range(t1, cols, wpr).first_float;
    const int nf = int(f1 - f0);  // <= 6 * 256
    for (int i = threadIdx.x; i < nf; i += kWordsPerBlock) {
        const float v = w[f0 + i];
        codes[i] = uint8_t(PS ? code_ps(v, sgn[f0 + i], max_shift) : code_q(v, max_shift));
    }
    __syncthreads();
    const int64_t t = t0 + threadIdx.x;
    if (t >= t1) return;
    const WordRange r = word_range(t, cols, wpr);
    const int base = int(r.first_float - f0);
    uint32_t word = 0;
    for (int i = 0; i < kCodesPerWord; ++i) {
        const uint32_t c = i < r.ncodes ? uint32_t(codes[base + i]) : kZeroCode;
        word |= c << (5 * i);
    }
    out[t] = word;
}

// round(x * 2^F) with halves away from zero, saturated to int32; NaN -> 0.
// x * 2^F is exact in float (a power-of-two scale) unless it overflows to inf,
// which saturates.
__device__ __forceinline__ int32_t to_fixed(float x, float scale)
{
    const float t = roundf(x * scale);
    if (t != t) return 0;
    if (t >= 2147483648.0f) return 2147483647;
    if (t < -2147483648.0f) return int32_t(0x80000000u);
    return int32_t(t);
}

constexpr int kFixedThreads = 256;

// Four elements per thread with one 16-byte load and store when both buffers
// are 16-byte aligned (the host checks); element-wise otherwise.
template <bool VEC>
__global__ __launch_bounds__(kFixedThreads) void to_fixed_kernel(
    const float *x, int64_t n, float scale, int32_t *y)  // x == y is allowed
{
    const int64_t stride = int64_t(gridDim.x) * kFixedThreads * 4;
    for (int64_t i = (int64_t(blockIdx.x) * kFixedThreads + threadIdx.x) * 4; i < n; i += stride) {
        if (VEC && i + 4 <= n) {
            const float4 v = *reinterpret_cast<const float4 *>(x + i);
            int4 o;
            o.x = to_fixed(v.x, scale);
            o.y = to_fixed(v.y, scale);
            o.z = to_fixed(v.z, scale);
            o.w = to_fixed(v.w, scale);
            *reinterpret_cast<int4 *>(y + i) = o;
        } else {
            for (int64_t j = i; j < min<int64_t>(i + 4, n); ++j)
                y[j] = to_fixed(x[j], scale);
        }
    }
}

ds_status hip_result(hipError_t e, const char *what)
{
    if (e == hipSuccess) return ok();
    return fail(DS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

ds_status check_quantize(const float *a, const float *b, bool need_b, int64_t rows, int64_t cols,
                         int32_t max_shift, const uint32_t *out, uint32_t flags, int64_t &nwords)
{
    if (!a || (need_b && !b) || !out) return fail(DS_ERR_NULL_POINTER, "inputs and output must not be NULL");
    if (rows <= 0 || cols <= 0) return fail(DS_ERR_INVALID_SHAPE, "rows and cols must be > 0");
    if (max_shift < 0 || max_shift > 14) return fail(DS_ERR_INVALID_ARG, "max_shift must be in [0, 14]");
    if (flags != 0) return fail(DS_ERR_INVALID_ARG, "flags must be 0");
    const int64_t ne = prod({rows, cols});
    nwords = prod({rows, row_words(cols)});
    if (ne < 0 || ne > kMaxElems || nwords < 0 || nwords > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    const int64_t ib = 4 * ne, ob = 4 * nwords;
    if (overlap(out, ob, a, ib) || (need_b && overlap(out, ob, b, ib)))
        return fail(DS_ERR_INVALID_ARG, "output overlaps an input");
    if (!device_range_ok(a, ib) || (need_b && !device_range_ok(b, ib)))
        return fail(DS_ERR_INVALID_ARG, "inputs are not device buffers of %lld bytes", (long long)ib);
    if (!device_range_ok(out, ob))
        return fail(DS_ERR_INVALID_ARG, "output is not a device buffer of %lld bytes", (long long)ob);
    return DS_SUCCESS;
}

template <bool PS>
ds_status launch_quantize(const float *a, const float *b, int64_t cols, int64_t nwords,
                          int32_t max_shift, uint32_t *out, void *stream, const char *name)
{
    const int64_t blocks = (nwords + kWordsPerBlock - 1) / kWordsPerBlock;
    hipLaunchKernelGGL(quantize_kernel<PS>, dim3(unsigned(blocks)), dim3(kWordsPerBlock), 0,
                       static_cast<hipStream_t>(stream), a, b, cols, row_words(cols), nwords,
                       int(max_shift), out);
    return hip_result(hipGetLastError(), name);
}

}  // namespace

}  // namespace ds

using namespace ds;

extern "C" ds_status ds_quantize_shift_weights_q(const float *w, int64_t rows, int64_t cols,
                                                 int32_t max_shift, uint32_t *w_packed,
                                                 uint32_t flags, void *stream)
{
    int64_t nwords = 0;
    const ds_status st = check_quantize(w, nullptr, false, rows, cols, max_shift, w_packed, flags, nwords);
    if (st != DS_SUCCESS) return st;
    return launch_quantize<false>(w, nullptr, cols, nwords, max_shift, w_packed, stream,
                                  "ds_quantize_shift_weights_q");
}

extern "C" ds_status ds_quantize_shift_weights_ps(const float *p, const float *s, int64_t rows,
                                                  int64_t cols, int32_t max_shift,
                                                  uint32_t *w_packed, uint32_t flags, void *stream)
{
    int64_t nwords = 0;
    const ds_status st = check_quantize(p, s, true, rows, cols, max_shift, w_packed, flags, nwords);
    if (st != DS_SUCCESS) return st;
    return launch_quantize<true>(p, s, cols, nwords, max_shift, w_packed, stream,
                                 "ds_quantize_shift_weights_ps");
}

extern "C" ds_status ds_to_fixed_point(const float *x, int64_t n, int32_t frac_bits, int32_t *y,
                                       uint32_t flags, void *stream)
{
    if (!x || !y) return fail(DS_ERR_NULL_POINTER, "x and y must not be NULL");
    if (n <= 0) return fail(DS_ERR_INVALID_SHAPE, "n must be > 0");
    if (n > kMaxElems) return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    if (frac_bits < 0 || frac_bits > 31) return fail(DS_ERR_INVALID_ARG, "frac_bits must be in [0, 31]");
    if (flags != 0) return fail(DS_ERR_INVALID_ARG, "flags must be 0");
    const int64_t bytes = 4 * n;
    if (overlap(x, bytes, y, bytes) && static_cast<const void *>(x) != static_cast<const void *>(y))
        return fail(DS_ERR_INVALID_ARG, "y partially overlaps x");
    if (!device_range_ok(x, bytes)) return fail(DS_ERR_INVALID_ARG, "x is not a device buffer of %lld bytes", (long long)bytes);
    if (!device_range_ok(y, bytes)) return fail(DS_ERR_INVALID_ARG, "y is not a device buffer of %lld bytes", (long long)bytes);
    const float scale = std::ldexp(1.0f, frac_bits);
    const int64_t groups = (n + 3) / 4;
    const int64_t blocks = std::min<int64_t>((groups + kFixedThreads - 1) / kFixedThreads, 8192);
    const bool vec = (reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y)) % 16 == 0;
    if (vec)
        hipLaunchKernelGGL(to_fixed_kernel<true>, dim3(unsigned(blocks)), dim3(kFixedThreads), 0,
                           static_cast<hipStream_t>(stream), x, n, scale, y);
    else
        hipLaunchKernelGGL(to_fixed_kernel<false>, dim3(unsigned(blocks)), dim3(kFixedThreads), 0,
                           static_cast<hipStream_t>(stream), x, n, scale, y);
    return hip_result(hipGetLastError(), "ds_to_fixed_point");
}
