// Input gradients of the shift operators (DeepShift Section 3, backward pass):
// the output gradient dY times the same quantised weights, i.e. the adjoint of
// the forward convolution (the footnote's convolution of dY with the weights
// rotated by 180 degrees), with the forward pass's shift terms:
//     dx[n][c][ih][iw] = sum over every (k, oh, ow, r, s) with
//                        oh*sh - ph + r == ih and ow*sw - pw + s == iw of
//                        term(dy[n][k][oh][ow], code[k][c][r][s])      (mod 2^32)
//
// Stride phases. For a stride (sh, sw) the rows ih = a + sh*i (a < sh) receive
// only the taps r = r0 + sh*t with r0 = (a + ph) mod sh, from the outputs
// oh = i + q - t with q = (a + ph - r0) / sh. Listing those taps in reverse
// order (t' = Ta - 1 - t) makes each phase (a, b) an ordinary stride-1
// correlation of dy with a Ta x Tb window, top padding pt = Ta - 1 - q (left
// likewise), whose outputs land on a regular sub-grid of dx. Each phase runs
// on the forward tiled kernel: its codes are re-packed (rows = input channels
// c, columns = (k, t', u') in the kernel's reduction order), and an output map
// places output (n, c, i, j) at dx[n][c][a + sh*i][b + sw*j]. Phases without
// taps are zero. A stride-1 layer is a single phase (the rotated, transposed
// kernel with padding R - 1 - p), and LinearShift the 1 x 1 case of it.
// Shapes the tiled kernel cannot take (a phase with negative padding, i.e.
// padding beyond the window, or no instance for its window width) use a
// one-thread-per-element gather kernel instead.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "common.hpp"
#include "conv_plan.hpp"

namespace ds {
namespace {

// One axis of a stride phase.
struct Axis {
    int out = 0;   // dx rows (or columns) in the phase
    int first = 0; // first tap of the phase (r0)
    int taps = 0;  // taps of the phase (Ta)
    int pad = 0;   // leading padding of the phase's stride-1 problem (may be < 0)
    int ext = 0;   // padded extent the phase's window staging needs
};

Axis phase_axis(int in, int out_fwd, int R, int stride, int pad, int a)
{
    Axis ax;
    ax.out = a < in ? (in - a + stride - 1) / stride : 0;
    ax.first = (a + pad) % stride;
    ax.taps = ax.first < R ? (R - ax.first + stride - 1) / stride : 0;
    const int q = (a + pad - ax.first) / stride;
    ax.pad = ax.taps - 1 - q;
    // the last output's window ends at padded row out - 1 + taps - 1
    ax.ext = std::max(ax.pad + out_fwd, ax.out - 1 + ax.taps);
    return ax;
}

}  // namespace

std::vector<GradPhase> grad_phases(const ConvGeom &g)
{
    std::vector<GradPhase> out;
    const bool single = g.sh == 1 && g.sw == 1;
    for (int a = 0; a < g.sh; ++a)
        for (int b = 0; b < g.sw; ++b) {
            const Axis ah = phase_axis(g.h, g.oh, g.r, g.sh, g.ph, a);
            const Axis aw = phase_axis(g.w, g.ow, g.s, g.sw, g.pw, b);
            if (ah.out == 0 || aw.out == 0) continue;  // no dx positions
            GradPhase p;
            p.a = a;
            p.b = b;
            p.r0 = ah.first;
            p.s0 = aw.first;
            p.ext_h = ah.ext;
            p.ext_w = aw.ext;
            ConvGeom &q = p.g;
            q.n = g.n; q.c = g.k; q.h = g.oh; q.w = g.ow; q.k = g.c;
            q.r = ah.taps; q.s = aw.taps; q.sh = 1; q.sw = 1;
            q.ph = ah.pad; q.pw = aw.pad; q.oh = ah.out; q.ow = aw.out;
            q.crs = g.k * q.r * q.s;
            q.bits = 5;
            if (!single) {
                p.map.base = int64_t(a) * g.w + b;
                p.map.nstride = g.c * g.h * g.w;
                p.map.kstride = g.h * g.w;
                p.map.rstride = g.sh * g.w;
                p.map.cstride = g.sw;
            }
            out.push_back(p);
        }
    return out;
}

namespace {

// Packed codes of one phase: row c, column j = (k * Ta + t) * Tb + u holds
// code[k][c][r0 + sh*(Ta-1-t)][s0 + sw*(Tb-1-u)] of the forward weights; the
// row is padded with code 15 to whole words.
__global__ void __launch_bounds__(256)
repack_phase_kernel(const uint32_t *__restrict__ wp, CodeFmt fmt, int K, int C, int R, int S,
                    int wpr, int r0, int s0, int sh, int sw, int Ta, int Tb, int wpr_out,
                    uint32_t *__restrict__ out)
{
    const int64_t total = int64_t(C) * wpr_out;
    const int per_k = Ta * Tb, cols = K * per_k;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int c = int(idx / wpr_out);
        const int wd = int(idx - int64_t(c) * wpr_out);
        uint32_t word = 0;
        for (int j = 0; j < 6; ++j) {
            const int jp = wd * 6 + j;
            uint32_t code = 15u;
            if (jp < cols) {
                const int k = jp / per_k, rem = jp - k * per_k;
                const int t = rem / Tb, u = rem - t * Tb;
                const int r = r0 + sh * (Ta - 1 - t), s = s0 + sw * (Tb - 1 - u);
                const int col = (c * R + r) * S + s;
                code = fmt.at(wp + int64_t(k) * wpr, col);
            }
            word |= code << (5 * j);
        }
        out[idx] = word;
    }
}

// One thread per dx element: every (k, r, s) whose forward output covers it.
__global__ void __launch_bounds__(256)
bwd_direct_kernel(const int32_t *__restrict__ dy, const uint32_t *__restrict__ wp,
                  int32_t *__restrict__ dx, ConvGeom g, int wpr, CodeFmt fmt)
{
    const int64_t total = int64_t(g.n) * g.c * g.h * g.w;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int iw = int(idx % g.w);
        int64_t t = idx / g.w;
        const int ih = int(t % g.h);
        t /= g.h;
        const int c = int(t % g.c);
        const int n = int(t / g.c);
        uint32_t acc = 0u;
        for (int k = 0; k < g.k; ++k)
            for (int r = 0; r < g.r; ++r) {
                const int a = ih + g.ph - r;  // = oh * sh
                if (a < 0 || a % g.sh != 0 || a / g.sh >= g.oh) continue;
                const int oh = a / g.sh;
                for (int s = 0; s < g.s; ++s) {
                    const int b = iw + g.pw - s;
                    if (b < 0 || b % g.sw != 0 || b / g.sw >= g.ow) continue;
                    const int32_t gv = dy[((int64_t(n) * g.k + k) * g.oh + oh) * g.ow + b / g.sw];
                    const int j = (c * g.r + r) * g.s + s;
                    const uint32_t code = fmt.at(wp + int64_t(k) * wpr, j);
                    const int sh = int(code & 15u);
                    if (sh == 15) continue;
                    const uint32_t tv = uint32_t(gv >> sh);
                    acc += (code & 16u) ? 0u - tv : tv;
                }
            }
        dx[idx] = int32_t(acc);
    }
}

struct PhasePlan {
    GradPhase ph;
    Padded pad;
    size_t word_offset;  // its re-packed codes in the scratch buffer
    int wpr;
};

// Phases of the input gradient of forward geometry g for the tiled kernel;
// false when one of them does not fit it.
bool plan_phases(const ConvGeom &g, std::vector<PhasePlan> &out, size_t &words)
{
    out.clear();
    words = 0;
    const bool single = g.sh == 1 && g.sw == 1;
    for (const GradPhase &ph : grad_phases(g)) {
        PhasePlan p;
        p.ph = ph;
        p.wpr = 0;
        const ConvGeom &q = ph.g;
        if (q.r > 0 && q.s > 0) {
            if (q.ph < 0 || q.pw < 0) return false;
            if (ph.ext_h != q.h + 2 * q.ph || ph.ext_w != q.w + 2 * q.pw) {
                if (single) return false;   // keeps the single phase on the dense path
                p.pad.vh = ph.ext_h;
                p.pad.iwp = ph.ext_w;
            }
            if (!tiled_fits(q, p.pad)) return false;
            p.wpr = int(row_words(q.crs));
            p.word_offset = words;
            words += (size_t(q.k) * p.wpr + 63) / 64 * 64;
        }
        out.push_back(p);
    }
    return true;
}

hipError_t run_backward_data(const ConvGeom &g, const int32_t *dy, const uint32_t *wp, int32_t *dx,
                             hipStream_t st)
{
    std::vector<PhasePlan> phases;
    size_t words = 0;
    const int wpr = int(row_words_bits(g.crs, g.bits));
    const CodeFmt fmt = code_fmt(g.bits);
    if (!plan_phases(g, phases, words) || forced_variant() == 0) {
        const int64_t total = int64_t(g.n) * g.c * g.h * g.w;
        const int grid = int(std::min<int64_t>((total + 255) / 256, 1 << 20));
        hipLaunchKernelGGL(bwd_direct_kernel, dim3(grid), dim3(256), 0, st, dy, wp, dx, g, wpr, fmt);
        return hipGetLastError();
    }
    void *scratch = nullptr;
    hipError_t e = words ? scratch_alloc(&scratch, words * 4, st) : hipSuccess;
    if (e != hipSuccess) return e;
    uint32_t *packed = static_cast<uint32_t *>(scratch);
    // Rows or columns no tap reaches are zero: dx is cleared densely first (the
    // phases then write their own positions), which is several times faster than
    // filling the empty phases through their strided maps.
    for (const PhasePlan &pp : phases)
        if (e == hipSuccess && (pp.ph.g.r == 0 || pp.ph.g.s == 0)) {
            e = run_fill_zero(dx, int64_t(g.n) * g.c * g.h * g.w, st);
            break;
        }
    for (const PhasePlan &pp : phases) {
        if (e != hipSuccess) break;
        const GradPhase &p = pp.ph;
        if (p.g.r == 0 || p.g.s == 0) continue;
        uint32_t *pw = packed + pp.word_offset;
        const int64_t total = int64_t(p.g.k) * pp.wpr;
        const int grid = int(std::min<int64_t>((total + 255) / 256, 4096));
        hipLaunchKernelGGL(repack_phase_kernel, dim3(grid), dim3(256), 0, st, wp, fmt, g.k, g.c, g.r,
                           g.s, wpr, p.r0, p.s0, g.sh, g.sw, p.g.r, p.g.s, pp.wpr, pw);
        e = hipGetLastError();
        if (e == hipSuccess)
            e = run_conv(p.g, dy, pw, nullptr, nullptr, dx, Inner::Shift, st, Epilogue(), p.map,
                         pp.pad);
    }
    const hipError_t ef = scratch ? hipFreeAsync(scratch, st) : hipSuccess;
    return e != hipSuccess ? e : ef;
}

void describe_backward(const ConvGeom &g, char *buf, size_t len)
{
    std::vector<PhasePlan> phases;
    size_t words = 0;
    if (!plan_phases(g, phases, words) || forced_variant() == 0) {
        snprintf(buf, len, "direct");
        return;
    }
    size_t used = size_t(snprintf(buf, len, "phases%zu", phases.size()));
    for (const PhasePlan &pp : phases) {
        if (used >= len) break;
        const ConvGeom &q = pp.ph.g;
        char sub[96];
        if (q.r == 0 || q.s == 0)
            snprintf(sub, sizeof sub, "zero");
        else
            describe_conv(q, sub, sizeof sub);
        used += size_t(snprintf(buf + used, len - used, "%s%dx%d %s", used ? "; " : "", q.r,
                                q.s, sub));
    }
}

// Validates a backward problem given by its forward geometry.
ds_status check_backward(const void *dy, const void *wp, const void *dx, int64_t n, int64_t c,
                         int64_t h, int64_t w, int64_t k, int64_t r, int64_t s, int32_t sh,
                         int32_t sw, int32_t ph, int32_t pw, int32_t frac_bits, uint32_t flags,
                         ConvGeom &g)
{
    if (!dy || !wp || !dx) return fail(DS_ERR_NULL_POINTER, "dy, w_packed and dx must not be NULL");
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0 || k <= 0 || r <= 0 || s <= 0)
        return fail(DS_ERR_INVALID_SHAPE, "all sizes must be > 0");
    if (sh < 1 || sw < 1) return fail(DS_ERR_INVALID_ARG, "stride must be >= 1");
    if (ph < 0 || pw < 0) return fail(DS_ERR_INVALID_ARG, "padding must be >= 0");
    if (h + 2 * int64_t(ph) < r || w + 2 * int64_t(pw) < s)
        return fail(DS_ERR_INVALID_SHAPE, "kernel larger than the padded input");
    if (frac_bits < 0 || frac_bits > 31) return fail(DS_ERR_INVALID_ARG, "frac_bits must be in [0, 31]");
    const int bits = flags_code_bits(flags);
    if ((flags & ~0xF00u) != 0 || bits < 0)
        return fail(DS_ERR_INVALID_ARG, "flags must be 0 apart from DS_CODE_BITS(2..5)");
    const int64_t oh = (h + 2 * int64_t(ph) - r) / sh + 1;
    const int64_t ow = (w + 2 * int64_t(pw) - s) / sw + 1;
    const int64_t crs = prod({c, r, s});
    const int64_t xe = prod({n, c, h, w}), ye = prod({n, k, oh, ow});
    const int64_t we = prod({k, row_words_bits(crs, bits)});
    if (crs < 0 || xe < 0 || ye < 0 || we < 0 || crs > kMaxElems || xe > kMaxElems ||
        ye > kMaxElems || we > kMaxElems || prod({k, crs}) > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    g = ConvGeom{int(n), int(c), int(h), int(w), int(k), int(r), int(s), sh, sw, ph, pw,
                 int(oh), int(ow), int(crs), bits};
    const int64_t dyb = 4 * ye, dxb = 4 * xe, wb = 4 * we;
    if (overlap(dx, dxb, dy, dyb) || overlap(dx, dxb, wp, wb))
        return fail(DS_ERR_INVALID_ARG, "dx overlaps an input");
    if (!device_range_ok(dy, dyb)) return fail(DS_ERR_INVALID_ARG, "dy is not a device buffer of %lld bytes", (long long)dyb);
    if (!device_range_ok(wp, wb)) return fail(DS_ERR_INVALID_ARG, "weights are not a device buffer of %lld bytes", (long long)wb);
    if (!device_range_ok(dx, dxb)) return fail(DS_ERR_INVALID_ARG, "dx is not a device buffer of %lld bytes", (long long)dxb);
    return DS_SUCCESS;
}

}  // namespace
}  // namespace ds

using namespace ds;

extern "C" ds_status ds_conv2d_shift_backward_data(const int32_t *dy, const uint32_t *w_packed,
                                                   int32_t *dx, int64_t n, int64_t c, int64_t h,
                                                   int64_t w, int64_t k, int64_t r, int64_t s,
                                                   int32_t stride_h, int32_t stride_w,
                                                   int32_t pad_h, int32_t pad_w, int32_t frac_bits,
                                                   uint32_t flags, void *stream)
{
    ConvGeom g;
    ds_status st = check_backward(dy, w_packed, dx, n, c, h, w, k, r, s, stride_h, stride_w, pad_h,
                                  pad_w, frac_bits, flags, g);
    if (st != DS_SUCCESS) return st;
    const hipError_t e = run_backward_data(g, dy, w_packed, dx, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(DS_ERR_HIP, "ds_conv2d_shift_backward_data: %s", hipGetErrorString(e));
    return ok();
}

extern "C" ds_status ds_linear_shift_backward_data(const int32_t *dy, const uint32_t *w_packed,
                                                   int32_t *dx, int64_t batch, int64_t in_features,
                                                   int64_t out_features, int32_t frac_bits,
                                                   uint32_t flags, void *stream)
{
    ConvGeom g;
    ds_status st = check_backward(dy, w_packed, dx, batch, in_features, 1, 1, out_features, 1, 1,
                                  1, 1, 0, 0, frac_bits, flags, g);
    if (st != DS_SUCCESS) return st;
    const hipError_t e = run_backward_data(g, dy, w_packed, dx, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(DS_ERR_HIP, "ds_linear_shift_backward_data: %s", hipGetErrorString(e));
    return ok();
}

extern "C" ds_status ds_conv2d_shift_backward_data_describe(int64_t n, int64_t c, int64_t h,
                                                            int64_t w, int64_t k, int64_t r,
                                                            int64_t s, int32_t stride_h,
                                                            int32_t stride_w, int32_t pad_h,
                                                            int32_t pad_w, char *buf, int64_t len)
{
    if (!buf) return fail(DS_ERR_NULL_POINTER, "buf must not be NULL");
    if (len < 1) return fail(DS_ERR_BUFFER_TOO_SMALL, "len must be >= 1");
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0 || k <= 0 || r <= 0 || s <= 0)
        return fail(DS_ERR_INVALID_SHAPE, "all sizes must be > 0");
    if (stride_h < 1 || stride_w < 1 || pad_h < 0 || pad_w < 0)
        return fail(DS_ERR_INVALID_ARG, "stride must be >= 1 and padding >= 0");
    if (h + 2 * int64_t(pad_h) < r || w + 2 * int64_t(pad_w) < s)
        return fail(DS_ERR_INVALID_SHAPE, "kernel larger than the padded input");
    const int64_t oh = (h + 2 * int64_t(pad_h) - r) / stride_h + 1;
    const int64_t ow = (w + 2 * int64_t(pad_w) - s) / stride_w + 1;
    if (prod({n, c, h, w}) > kMaxElems || prod({n, k, oh, ow}) > kMaxElems || prod({c, r, s}) > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors with 2^31 or more elements are not supported");
    const ConvGeom g{int(n), int(c), int(h), int(w), int(k), int(r), int(s), stride_h, stride_w,
                     pad_h, pad_w, int(oh), int(ow), int(c * r * s)};
    describe_backward(g, buf, size_t(len));
    return ok();
}
