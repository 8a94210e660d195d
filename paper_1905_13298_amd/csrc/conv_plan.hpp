// Problem geometry and the launch entry shared by the operator front ends.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "common.hpp"

namespace ds {

// One convolution problem (LinearShift is the case h = w = r = s = 1).
struct ConvGeom {
    int n, c, h, w, k, r, s;
    int sh, sw, ph, pw;
    int oh, ow;
    int crs;
    int bits = 5;  // width of the packed weight codes
};

// Inner operation of the reduction: the DeepShift shift-accumulate, or the
// multiplication-based comparison: int32 multiply-add, or the multiply-add of
// the low 24 bits of both operands taken as signed (v_mad_i32_i24), equal to the
// int32 one while |x| and |w| are below 2^23.
enum class Inner { Shift, Mul, Mul24 };

// The product of the comparison operator Mul24: sext(a[23:0]) * sext(b[23:0]) mod 2^32.
DS_HD inline uint32_t mul24(int32_t a, int32_t b)
{
    const int32_t a24 = int32_t(uint32_t(a) << 8) >> 8, b24 = int32_t(uint32_t(b) << 8) >> 8;
    return uint32_t(a24) * uint32_t(b24);
}

// What follows the convolution on each output y[n][k][p] (all optional):
//   v = floor(v * mul[k] / 2^mul_shift) + add[k]   (when mul; add may be NULL)
//   v = v + res[n][k][p]                           (when res)
//   v = max(v, 0)                                  (when relu)
// with int32 wrap-around, as in the accumulation.
struct Epilogue {
    const int32_t *mul = nullptr, *add = nullptr, *res = nullptr;
    int mul_shift = 0;
    bool relu = false;
    bool any() const { return mul || res || relu; }
};

// Where output (n, k, oh, ow) of a problem lands in y:
//     y[base + n * nstride + k * kstride + oh * rstride + ow * cstride]
// The default (all zero) is the dense NCHW layout of the problem's own output.
// A strided map lets one problem fill a regular sub-grid of a larger tensor
// (the stride phases of an input gradient).
struct OutMap {
    int64_t base = 0;
    int nstride = 0, kstride = 0, rstride = 0, cstride = 0;
    bool dense() const { return nstride == 0; }
};

// Padded extents of the input in the window staging mode: `vh` rows (top
// padding ph, then h rows, then whatever bottom padding reaches vh) and `iwp`
// columns per row. Zero means the symmetric default h + 2 ph, w + 2 pw.
struct Padded {
    int vh = 0, iwp = 0;
};

// Device memory a call may use for its scratch instead of allocating it: at
// `ptr`, `bytes` long, 256-byte aligned (ptr == nullptr: allocate in stream order).
struct Workspace {
    void *ptr = nullptr;
    size_t bytes = 0;
};

// Enqueue the whole computation of y on `stream`. Exactly one of `wpacked`
// (Shift) and `wint` (Mul) is used. g.oh and g.ow give the output grid; with
// the defaults of `map` and `pad` they must be the usual output sizes. With a
// workspace of at least conv_scratch_bytes(g, map, pad) bytes the call
// allocates nothing; a smaller one fails with hipErrorInvalidValue before any
// launch.
hipError_t run_conv(const ConvGeom &g, const int32_t *x, const uint32_t *wpacked,
                    const int32_t *wint, const int32_t *bias, int32_t *y, Inner op,
                    hipStream_t stream, const Epilogue &epi = Epilogue(),
                    const OutMap &map = OutMap(), const Padded &pad = Padded(),
                    const Workspace &ws = Workspace());

// Scratch bytes run_conv takes for g (0 when it runs the one-thread-per-output
// kernel, which needs none). Host only; touches no device.
size_t conv_scratch_bytes(const ConvGeom &g, const OutMap &map = OutMap(),
                          const Padded &pad = Padded());

// One stride phase of the input gradient of a forward layer (backward.hip): the
// stride-1 correlation of dy that produces the dx rows a + sh*i and columns
// b + sw*j, with the phase's taps in reverse order.
struct GradPhase {
    ConvGeom g;        // the phase's problem: input dy [n][k][oh][ow], output channels c
    OutMap map;        // its place in dx (the dense default for a stride-1 layer)
    int a, b;          // row and column residues
    int r0, s0;        // first forward tap row and column of the phase
    int ext_h, ext_w;  // padded extents the phase's window staging needs
};

// The phases of the input gradient of forward layer g, in (a, b) order, leaving
// out residues with no dx positions; a phase that no tap reaches has g.r == 0
// or g.s == 0 (its dx positions are zero).
std::vector<GradPhase> grad_phases(const ConvGeom &g);

// Whether run_conv runs g (with `pad`) on the tiled kernel rather than the
// one-thread-per-output kernel.
bool tiled_fits(const ConvGeom &g, const Padded &pad);

// Stream-ordered device scratch from the library's memory pool.
hipError_t scratch_alloc(void **p, size_t bytes, hipStream_t stream);

// y[n][k][p] = init[k] (the start of split-K accumulation), and the epilogue as
// a pass of its own over y, both enqueued on `stream`.
hipError_t run_fill_init(const ConvGeom &g, const int32_t *init, int32_t *y, hipStream_t stream);
// The same through a map; init == NULL writes zeros.
hipError_t run_fill_mapped(const ConvGeom &g, const int32_t *init, int32_t *y, const OutMap &map,
                           hipStream_t stream);
// y[map(n, k, oh, ow)] = src (dense [n][k][oh][ow]) for a strided map.
hipError_t run_copy_mapped(const ConvGeom &g, const int32_t *src, int32_t *y, const OutMap &map,
                           hipStream_t stream);
hipError_t run_epilogue(const ConvGeom &g, int32_t *y, const Epilogue &epi, hipStream_t stream);
// y[0 .. count) = 0 (a 4-byte-aligned y), in 16-byte stores where aligned.
hipError_t run_fill_zero(int32_t *y, int64_t count, hipStream_t stream);
// xp [planes][xh][xw] = x [planes][h][w] shifted down by ph rows and right by pw
// columns, zeros elsewhere (rows and columns past xh, xw are dropped); x holds
// xbytes-byte signed integers (4, 2 or 1), xp int32 (sign-extended).
hipError_t run_pad_planes(const void *x, int32_t *xp, int64_t planes, int h, int w, int ph,
                          int pw, int xh, int xw, hipStream_t stream, int xbytes = 4);


// Short name of the kernel run_conv would launch for g (see ds_conv2d_shift_describe).
void describe_conv(const ConvGeom &g, char *buf, size_t len);

// Kernel variant forced for testing and tuning (the DS_FORCE_VARIANT knob of
// tuning.hpp): -1 = automatic choice, 0 = the one-thread-per-output kernel,
// 8 = tiled kernels with 8 pixels per lane where an instance exists (the
// default is 4).
int forced_variant();

}  // namespace ds
