// Float -> shift-code converter and float -> fixed-point conversion, the steps
// that feed the shift operators:
//   * DeepShift-Q (Section 3, Eqs. 4-5): sign(w) and round(log2|w|);
//   * DeepShift-PS (Section 3): round(P) and the ternary sign thresholds +-0.5;
//   * the power is clipped to -max_shift .. 0 (Section 4, 14 for 5-bit codes);
//   * inputs and bias rounded to fixed point with F fractional bits
//     (Section 4, 16.16).
// The weight converters write the packed format directly: 5-bit codes, or the
// shorter b-bit codes of DS_CODE_BITS (Section 5's shorter shift ranges).
//
// Both are streaming kernels bound by HBM bandwidth. A weight block owns 256
// consecutive packed words. The floats those words cover form one contiguous
// range (rows are stored back to back), so the block reads that range with
// coalesced loads, turns every float into its code once, keeps the codes as
// bytes in LDS, and then each thread gathers the codes of its word (six for
// 5-bit codes, floor(32 / b) for b bits) and stores the word (coalesced).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <string>

#include "common.hpp"
#include "fastdiv.hpp"

namespace ds {

namespace {

constexpr int kWordsPerBlock = 256;
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
    int first_float;  // flat index (within the tensor) of the first float of word t
    int ncodes;       // codes of word t that come from the row (1..PER)
};

// Word t of a tensor with `cols` floats and `wpr` words per row, PER codes per
// word (all indexes below 2^31: the entry points reject larger tensors).
template <int PER>
__device__ __forceinline__ WordRange word_range(int t, int cols, const FastDiv &wpr)
{
    const int row = fdiv(t, wpr), j = t - row * int(wpr.d);
    const int col = j * PER;
    WordRange r;
    r.first_float = row * cols + col;
    r.ncodes = min(PER, cols - col);
    return r;
}

// A 5-bit code in the BITS-bit layout: the sign on top, the shift code below,
// all ones for a zero weight (the entry points keep max_shift inside the range).
template <int BITS>
__device__ __forceinline__ uint32_t narrow(uint32_t code)
{
    constexpr uint32_t ones = (1u << (BITS - 1)) - 1u;
    const uint32_t sh = code & 15u;
    return ((code >> 4) << (BITS - 1)) | (sh == 15u ? ones : sh);
}

// One weight tensor of a launch: its inputs, its packed output, and the first
// block of the launch that works on it.
struct Segment {
    const float *a;     // w (DeepShift-Q) or P (DeepShift-PS)
    const float *b;     // S (DeepShift-PS), unused otherwise
    uint32_t *out;
    int cols, nwords, rows;
    int block0;         // first block of the launch that works on this tensor
    FastDiv wpr;        // words per row
};

// Up to kMaxSegments tensors per launch, passed by value in the kernel
// arguments (about 3.5 KB, under the 4 KB limit), so a launch needs no device
// table.
constexpr int kMaxSegments = 64;
struct SegmentTable {
    int count;
    int max_shift;
    Segment seg[kMaxSegments];
};

template <bool PS, int BITS>
__global__ __launch_bounds__(kWordsPerBlock) void quantize_kernel(const SegmentTable tab)
{
    constexpr int PER = 32 / BITS;
    __shared__ uint8_t codes[kWordsPerBlock * PER];
    // This block's tensor: the last segment whose first block is <= blockIdx.x.
    int lo = 0, hi = tab.count - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tab.seg[mid].block0 <= int(blockIdx.x)) lo = mid; else hi = mid - 1;
    }
    const Segment &sg = tab.seg[lo];
    const int cols = sg.cols, nwords = sg.nwords;
    const int t0 = (int(blockIdx.x) - sg.block0) * kWordsPerBlock;
    const int t1 = min(t0 + kWordsPerBlock, nwords);
    // Floats covered by words [t0, t1): [f0, f1). Word t1 (or the end) starts at f1.
    const int f0 = word_range<PER>(t0, cols, sg.wpr).first_float;
    const int f1 = t1 == nwords ? sg.rows * cols : word_range<PER>(t1, cols, sg.wpr).first_float;
    const int nf = f1 - f0;  // <= PER * 256
    const float *__restrict__ a = sg.a + f0;
    const float *__restrict__ b = PS ? sg.b + f0 : nullptr;
    // PER independent loads per thread in flight, then the codes into LDS.
    float va[PER], vb[PER];
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int i = int(threadIdx.x) + r * kWordsPerBlock;
        va[r] = i < nf ? a[i] : 0.0f;
        vb[r] = PS && i < nf ? b[i] : 0.0f;
    }
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int i = int(threadIdx.x) + r * kWordsPerBlock;
        if (i < nf)
            codes[i] = uint8_t(PS ? code_ps(va[r], vb[r], tab.max_shift) : code_q(va[r], tab.max_shift));
    }
    __syncthreads();
    const int t = t0 + int(threadIdx.x);
    if (t >= t1) return;
    const WordRange r = word_range<PER>(t, cols, sg.wpr);
    const int base = int(r.first_float - f0);
    uint32_t word = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const uint32_t c = i < r.ncodes ? uint32_t(codes[base + i]) : kZeroCode;
        word |= narrow<BITS>(c) << (BITS * i);
    }
    sg.out[t] = word;
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

// The same rounding saturated to the range of T (int16 or int8): the lower
// bit-width activations of Section 5. Four elements per thread, with a 16-byte
// load and a 4 * sizeof(T)-byte store when both buffers are aligned for them.
template <typename T, bool VEC>
__global__ __launch_bounds__(kFixedThreads) void to_fixed_narrow_kernel(const float *x, int64_t n,
                                                                        float scale, T *y)
{
    constexpr int32_t lo = -(1 << (8 * sizeof(T) - 1)), hi = (1 << (8 * sizeof(T) - 1)) - 1;
    const int64_t stride = int64_t(gridDim.x) * kFixedThreads * 4;
    for (int64_t i = (int64_t(blockIdx.x) * kFixedThreads + threadIdx.x) * 4; i < n; i += stride) {
        if (VEC && i + 4 <= n) {
            const float4 v = *reinterpret_cast<const float4 *>(x + i);
            T o[4] = {T(min(max(to_fixed(v.x, scale), lo), hi)), T(min(max(to_fixed(v.y, scale), lo), hi)),
                      T(min(max(to_fixed(v.z, scale), lo), hi)), T(min(max(to_fixed(v.w, scale), lo), hi))};
            if constexpr (sizeof(T) == 2)
                *reinterpret_cast<short4 *>(y + i) = make_short4(o[0], o[1], o[2], o[3]);
            else
                *reinterpret_cast<char4 *>(y + i) = make_char4(o[0], o[1], o[2], o[3]);
        } else {
            for (int64_t j = i; j < min<int64_t>(i + 4, n); ++j)
                y[j] = T(min(max(to_fixed(x[j], scale), lo), hi));
        }
    }
}

ds_status hip_result(hipError_t e, const char *what)
{
    if (e == hipSuccess) return ok();
    return fail(DS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Argument checks of one tensor that need no device access.
ds_status check_quantize(const float *a, const float *b, bool need_b, int64_t rows, int64_t cols,
                         int32_t max_shift, const uint32_t *out, uint32_t flags, int64_t &nwords)
{
    if (!a || (need_b && !b) || !out) return fail(DS_ERR_NULL_POINTER, "inputs and output must not be NULL");
    if (rows <= 0 || cols <= 0) return fail(DS_ERR_INVALID_SHAPE, "rows and cols must be > 0");
    if (max_shift < 0 || max_shift > 14) return fail(DS_ERR_INVALID_ARG, "max_shift must be in [0, 14]");
    const int bits = flags_code_bits(flags);
    if ((flags & ~0xF00u) != 0 || bits < 0)
        return fail(DS_ERR_INVALID_ARG, "flags must be 0 apart from DS_CODE_BITS(2..5)");
    if (max_shift > (1 << (bits - 1)) - 2)
        return fail(DS_ERR_INVALID_ARG, "max_shift %d does not fit %d-bit codes (at most %d)",
                    int(max_shift), bits, (1 << (bits - 1)) - 2);
    const int64_t ne = prod({rows, cols});
    nwords = prod({rows, row_words_bits(cols, bits)});
    if (ne < 0 || ne > kMaxElems || nwords < 0 || nwords > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    const int64_t ib = 4 * ne, ob = 4 * nwords;
    if (overlap(out, ob, a, ib) || (need_b && overlap(out, ob, b, ib)))
        return fail(DS_ERR_INVALID_ARG, "output overlaps an input");
    return DS_SUCCESS;
}

// The buffers of one tensor must be device allocations of the required size.
ds_status check_quantize_buffers(const float *a, const float *b, bool need_b, int64_t rows,
                                 int64_t cols, const uint32_t *out, int bits)
{
    const int64_t ib = 4 * rows * cols, ob = 4 * rows * row_words_bits(cols, bits);
    if (!device_range_ok(a, ib) || (need_b && !device_range_ok(b, ib)))
        return fail(DS_ERR_INVALID_ARG, "inputs are not device buffers of %lld bytes", (long long)ib);
    if (!device_range_ok(out, ob))
        return fail(DS_ERR_INVALID_ARG, "output is not a device buffer of %lld bytes", (long long)ob);
    return DS_SUCCESS;
}

// Validates every tensor first (nothing is launched on an error), then
// launches once per kMaxSegments tensors.
template <bool PS>
ds_status quantize_many(int64_t count, const float *const *a, const float *const *b,
                        const int64_t *rows, const int64_t *cols, uint32_t *const *out,
                        int32_t max_shift, uint32_t flags, void *stream, const char *name)
{
    if (count <= 0) return fail(DS_ERR_INVALID_SHAPE, "count must be > 0");
    if (!a || (PS && !b) || !rows || !cols || !out)
        return fail(DS_ERR_NULL_POINTER, "the arrays must not be NULL");
    auto named = [&](ds_status st, int64_t i) {
        if (count == 1) return st;
        const std::string msg = last_error();
        return fail(st, "tensor %lld: %s", (long long)i, msg.c_str());
    };
    const int bits = flags_code_bits(flags);
    // Arguments of every tensor first, then the device buffers.
    for (int64_t i = 0; i < count; ++i) {
        int64_t nwords = 0;
        const ds_status st = check_quantize(a[i], PS ? b[i] : nullptr, PS, rows[i], cols[i],
                                            max_shift, out[i], flags, nwords);
        if (st != DS_SUCCESS) return named(st, i);
        for (int64_t j = 0; j < i; ++j)
            if (overlap(out[i], 4 * nwords, out[j], 4 * rows[j] * row_words_bits(cols[j], bits)) ||
                overlap(out[i], 4 * nwords, a[j], 4 * rows[j] * cols[j]) ||
                overlap(out[j], 4 * rows[j] * row_words_bits(cols[j], bits), a[i], 4 * rows[i] * cols[i]))
                return fail(DS_ERR_INVALID_ARG, "tensors %lld and %lld overlap (an output over "
                            "an input or another output)", (long long)j, (long long)i);
    }
    for (int64_t i = 0; i < count; ++i) {
        const ds_status st = check_quantize_buffers(a[i], PS ? b[i] : nullptr, PS, rows[i], cols[i],
                                                    out[i], bits);
        if (st != DS_SUCCESS) return named(st, i);
    }
    for (int64_t first = 0; first < count; first += kMaxSegments) {
        SegmentTable tab;
        tab.count = int(std::min<int64_t>(kMaxSegments, count - first));
        tab.max_shift = max_shift;
        int64_t blocks = 0;
        for (int i = 0; i < tab.count; ++i) {
            const int64_t k = first + i;
            Segment &sg = tab.seg[i];
            sg.a = a[k];
            sg.b = PS ? b[k] : nullptr;
            sg.out = out[k];
            sg.cols = int(cols[k]);
            sg.rows = int(rows[k]);
            sg.wpr = make_fastdiv(uint32_t(row_words_bits(cols[k], bits)));
            sg.nwords = int(rows[k] * row_words_bits(cols[k], bits));
            if (blocks > INT32_MAX) return fail(DS_ERR_UNSUPPORTED, "too many weights in one call");
            sg.block0 = int(blocks);
            blocks += (sg.nwords + kWordsPerBlock - 1) / kWordsPerBlock;
        }
        if (blocks > INT32_MAX) return fail(DS_ERR_UNSUPPORTED, "too many weights in one call");
        const hipStream_t st_ = static_cast<hipStream_t>(stream);
        const dim3 grid{unsigned(blocks)}, block{unsigned(kWordsPerBlock)};
        switch (bits) {
        case 2: hipLaunchKernelGGL((quantize_kernel<PS, 2>), grid, block, 0, st_, tab); break;
        case 3: hipLaunchKernelGGL((quantize_kernel<PS, 3>), grid, block, 0, st_, tab); break;
        case 4: hipLaunchKernelGGL((quantize_kernel<PS, 4>), grid, block, 0, st_, tab); break;
        default: hipLaunchKernelGGL((quantize_kernel<PS, 5>), grid, block, 0, st_, tab); break;
        }
        const ds_status st = hip_result(hipGetLastError(), name);
        if (st != DS_SUCCESS) return st;
    }
    return ok();
}

}  // namespace

}  // namespace ds

using namespace ds;

extern "C" ds_status ds_quantize_shift_weights_q(const float *w, int64_t rows, int64_t cols,
                                                 int32_t max_shift, uint32_t *w_packed,
                                                 uint32_t flags, void *stream)
{
    if (!w || !w_packed) return fail(DS_ERR_NULL_POINTER, "inputs and output must not be NULL");
    return quantize_many<false>(1, &w, nullptr, &rows, &cols, &w_packed, max_shift, flags, stream,
                                "ds_quantize_shift_weights_q");
}

extern "C" ds_status ds_quantize_shift_weights_ps(const float *p, const float *s, int64_t rows,
                                                  int64_t cols, int32_t max_shift,
                                                  uint32_t *w_packed, uint32_t flags, void *stream)
{
    if (!p || !s || !w_packed) return fail(DS_ERR_NULL_POINTER, "inputs and output must not be NULL");
    return quantize_many<true>(1, &p, &s, &rows, &cols, &w_packed, max_shift, flags, stream,
                               "ds_quantize_shift_weights_ps");
}

extern "C" ds_status ds_quantize_shift_weights_q_many(int64_t count, const float *const *w,
                                                      const int64_t *rows, const int64_t *cols,
                                                      int32_t max_shift, uint32_t *const *w_packed,
                                                      uint32_t flags, void *stream)
{
    return quantize_many<false>(count, w, nullptr, rows, cols, w_packed, max_shift, flags, stream,
                                "ds_quantize_shift_weights_q_many");
}

extern "C" ds_status ds_to_fixed_point(const float *x, int64_t n, int32_t frac_bits, void *yv,
                                       uint32_t flags, void *stream)
{
    int32_t *y = static_cast<int32_t *>(yv);  // int16 / int8 elements with DS_ACT_I16 / DS_ACT_I8
    if (!x || !y) return fail(DS_ERR_NULL_POINTER, "x and y must not be NULL");
    if (n <= 0) return fail(DS_ERR_INVALID_SHAPE, "n must be > 0");
    if (n > kMaxElems) return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    if (frac_bits < 0 || frac_bits > 31) return fail(DS_ERR_INVALID_ARG, "frac_bits must be in [0, 31]");
    if (flags != 0 && flags != DS_ACT_I16 && flags != DS_ACT_I8)
        return fail(DS_ERR_INVALID_ARG, "flags must be 0, DS_ACT_I16 or DS_ACT_I8");
    const int64_t bytes = 4 * n;
    const int64_t ybytes = flags == DS_ACT_I16 ? 2 * n : flags == DS_ACT_I8 ? n : bytes;
    if (overlap(x, bytes, y, ybytes) && (flags != 0 || static_cast<const void *>(x) != static_cast<const void *>(y)))
        return fail(DS_ERR_INVALID_ARG, flags ? "y overlaps x" : "y partially overlaps x");
    if (!device_range_ok(x, bytes)) return fail(DS_ERR_INVALID_ARG, "x is not a device buffer of %lld bytes", (long long)bytes);
    if (!device_range_ok(y, ybytes)) return fail(DS_ERR_INVALID_ARG, "y is not a device buffer of %lld bytes", (long long)ybytes);
    const float scale = std::ldexp(1.0f, frac_bits);
    const int64_t groups = (n + 3) / 4;
    const int64_t blocks = std::min<int64_t>((groups + kFixedThreads - 1) / kFixedThreads, 8192);
    if (flags != 0) {
        const int ysize = flags == DS_ACT_I16 ? 2 : 1;
        const bool v = reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(y) % (4 * ysize) == 0;
        hipStream_t st = static_cast<hipStream_t>(stream);
        if (ysize == 2 && v)
            hipLaunchKernelGGL((to_fixed_narrow_kernel<int16_t, true>), dim3(unsigned(blocks)), dim3(kFixedThreads), 0, st,
                               x, n, scale, static_cast<int16_t *>(static_cast<void *>(y)));
        else if (ysize == 2)
            hipLaunchKernelGGL((to_fixed_narrow_kernel<int16_t, false>), dim3(unsigned(blocks)), dim3(kFixedThreads), 0, st,
                               x, n, scale, static_cast<int16_t *>(static_cast<void *>(y)));
        else if (v)
            hipLaunchKernelGGL((to_fixed_narrow_kernel<int8_t, true>), dim3(unsigned(blocks)), dim3(kFixedThreads), 0, st,
                               x, n, scale, static_cast<int8_t *>(static_cast<void *>(y)));
        else
            hipLaunchKernelGGL((to_fixed_narrow_kernel<int8_t, false>), dim3(unsigned(blocks)), dim3(kFixedThreads), 0, st,
                               x, n, scale, static_cast<int8_t *>(static_cast<void *>(y)));
        return hip_result(hipGetLastError(), "ds_to_fixed_point");
    }
    const bool vec = (reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y)) % 16 == 0;
    if (vec)
        hipLaunchKernelGGL(to_fixed_kernel<true>, dim3(unsigned(blocks)), dim3(kFixedThreads), 0,
                           static_cast<hipStream_t>(stream), x, n, scale, y);
    else
        hipLaunchKernelGGL(to_fixed_kernel<false>, dim3(unsigned(blocks)), dim3(kFixedThreads), 0,
                           static_cast<hipStream_t>(stream), x, n, scale, y);
    return hip_result(hipGetLastError(), "ds_to_fixed_point");
}
