/*
 * deepshift.h -- C ABI of the DeepShift shift-operator library for AMD
 * Instinct MI355X (gfx950).
 *
 * The library computes the inference forward pass of the two DeepShift
 * operators, LinearShift and ConvShift (Elhoushi et al., "DeepShift: Towards
 * Multiplication-Less Neural Networks", Section 3). Every weight is
 * flip(2^p, s) (Eq. 3): a power of two p in {0, -1, ..., -14} and a ternary
 * sign s in {-1, 0, +1} (Eq. 2), stored in 5 bits (Section 4). Activations
 * and bias are fixed point (Section 4 uses 32 bits with 16 fractional bits).
 * Each multiply-accumulate becomes an arithmetic right shift, an optional
 * negation and an integer add (Figure 1a, Eq. 1).
 *
 * Exact semantics of one term (the readings this library takes where the
 * paper is silent):
 *     term(x, code) = 0                       if shift_code == 15
 *                   = -(x >> shift_code)      if sign bit set
 *                   =  (x >> shift_code)      otherwise
 * where ">>" is the arithmetic (flooring) right shift of a signed int32, and
 * outputs are  y = bias + sum of terms, computed modulo 2^32 (two's
 * complement wrap-around of int32). The result does not depend on the
 * number of fractional bits F: every weight is a dimensionless power of two
 * <= 1, so y carries the same F as x and bias.
 *
 * Weight codes (unpacked form, one uint8 per weight):
 *     bit 4    sign (1 = negative)
 *     bits 0-3 shift code: 0..14 means p = -code, 15 means a zero weight
 *              (whatever the sign bit)
 *     bits 5-7 must be 0
 * Packed form (what the compute entry points read): each weight row is
 * stored in ds_packed_row_words(cols) uint32 words, six codes per word, code
 * j of a word in bits [5j, 5j+5), bits 30-31 zero, and the last word of a row
 * filled up with code 15. Rows follow each other with no gap.
 *
 * Ownership and memory: the caller owns every buffer. Compute entry points
 * take device pointers on the current HIP device; the pack/unpack helpers
 * take host pointers. y must not overlap any input. The runtime-weights
 * entry points (ds_linear_shift, ds_conv2d_shift and their variants) take
 * device scratch memory (decoded weights, per-channel start values, transposed
 * operands; none for a LinearShift of fewer than 256 rows, whose kernel decodes
 * the packed codes itself) in stream order from the device's default memory pool
 * (hipMallocAsync) and give it back in stream order (hipFreeAsync) within the
 * same call: the library keeps no pool and no device memory between calls.
 * Under the runtime's default release threshold the memory returns to the
 * driver at the caller's next synchronisation. Callers that cannot allocate
 * use ds_conv2d_shift_noalloc (below). Plans (ds_jit_conv_*) hold the device
 * memory they need from create to destroy.
 *
 * Errors: arguments are validated before any device work. On a validation
 * error nothing is written and nothing is launched. Compute entry points are
 * asynchronous with respect to the host: they enqueue work on `stream`
 * (a hipStream_t; NULL = the default stream) and return. A failure reported
 * by the HIP runtime while enqueueing returns DS_ERR_HIP;
 * ds_last_error_message() then describes it. No exception crosses the ABI.
 */
#ifndef DEEPSHIFT_H
#define DEEPSHIFT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* flags bit of the shift operators: replace every output v by max(v, 0)
 * (ReLU fused into the operator, as Section 6 suggests). */
#define DS_RELU 1u

/* flags bit of ds_jit_conv_create: ds_jit_conv_run adds a residual tensor
 * (shape of y) after the affine map and before ReLU. */
#define DS_JIT_RESIDUAL 2u

/* flags field (bits 8-11) of every entry point that reads packed weights: the
 * width b of the packed codes, 2..5 (0 = 5). Section 4 keeps the weights in 5
 * bits (1 sign bit, a 4-bit shift) and Section 5 trains with fewer bits by
 * limiting the shifts to shorter ranges. A b-bit code holds the sign in its top
 * bit and a (b-1)-bit shift code below it, all ones meaning a zero weight, so
 * the shifts are 0 .. -(2^(b-1) - 2): 4 bits reach -6, 3 bits -2, and 2 bits
 * give the ternary weights {-1, 0, +1}. A row of `cols` codes takes
 * ds_packed_row_words_bits(cols, b) words, floor(32 / b) codes per word, code j
 * of a word in bits [b*j, b*j + b), unused top bits zero, the last word filled
 * with the zero code. For b = 5 this is the default layout described above. */
#define DS_CODE_BITS(b) ((uint32_t)(b) << 8)

/* flags field (bits 12-13) of ds_jit_conv_create and ds_to_fixed_point: the width
 * of the activations. Section 5 (lower bit-widths) trains with 16-bit activations
 * in fixed point with 3 integer and 13 fractional bits (3.13), and with 8-bit
 * ones; the text gives the same 3.13 split for 8 bits, which cannot fit, so this
 * library reads 8-bit activations as 3.5 (3 integer bits with the sign, 5
 * fractional). The library does not depend on the split: F is the caller's.
 * DS_ACT_I16: x is int16; DS_ACT_I8: x is int8 (0: int32). A shift of a
 * sign-extended value is the sign-extended shift, so every term and the int32
 * sum are those of the int32 operator on the sign-extended inputs; only the
 * bytes of x read from memory change. */
#define DS_ACT_I16 (1u << 12)
#define DS_ACT_I8 (2u << 12)

typedef enum ds_status {
    DS_SUCCESS = 0,
    DS_ERR_NULL_POINTER = 1,     /* a required pointer is NULL */
    DS_ERR_INVALID_SHAPE = 2,    /* a size is <= 0, or an output size would be <= 0 */
    DS_ERR_INVALID_ARG = 3,      /* bad stride/pad/frac_bits/flags, overlap, or a
                                    buffer that is not device memory of the size needed */
    DS_ERR_BUFFER_TOO_SMALL = 4, /* a host output buffer is shorter than required */
    DS_ERR_INVALID_CODE = 5,     /* a weight code >= 32 */
    DS_ERR_HIP = 6,              /* the HIP runtime reported an error */
    DS_ERR_UNSUPPORTED = 7,      /* a tensor has 2^31 or more elements */
    DS_STATUS_MAX_ = 0x7fffffff  /* not a status: widens the type to every int value, so that
                                    ds_status_string may be given any int */
} ds_status;

/* Number of uint32 words one packed row of `cols` codes occupies:
 * ceil(cols / 6). Returns -1 when cols <= 0. */
int64_t ds_packed_row_words(int64_t cols);

/* Pack host codes [rows][cols] (uint8, layout above) into host words
 * [rows][ds_packed_row_words(cols)] (the 5-bit weight format of Section 4).
 * packed_words is the capacity of `packed` in words.
 * Errors: NULL pointer, rows/cols <= 0, capacity too small, any code >= 32
 * (DS_ERR_INVALID_CODE, nothing written). */
ds_status ds_pack_shift_weights(const uint8_t *codes, int64_t rows, int64_t cols,
                                uint32_t *packed, int64_t packed_words);

/* Inverse of ds_pack_shift_weights (host memory). codes_len is the capacity
 * of `codes` in bytes. Words with bits 30-31 set give DS_ERR_INVALID_CODE. */
ds_status ds_unpack_shift_weights(const uint32_t *packed, int64_t rows, int64_t cols,
                                  uint8_t *codes, int64_t codes_len);

/* The b-bit packed format of DS_CODE_BITS (host memory), b in 2..5. The codes
 * are given and returned in the unpacked 5-bit form above; packing fails with
 * DS_ERR_INVALID_CODE (nothing written) when a code is >= 32 or its shift does
 * not fit b bits (a shift code above 2^(b-1) - 2 other than 15). Unpacking
 * returns canonical codes (a zero weight as shift code 15, its sign bit kept)
 * and fails when a word's unused top bits are set. ds_packed_row_words_bits
 * returns -1 for cols <= 0 or b outside 2..5. */
int64_t ds_packed_row_words_bits(int64_t cols, int32_t bits);
ds_status ds_pack_shift_weights_bits(const uint8_t *codes, int64_t rows, int64_t cols,
                                     int32_t bits, uint32_t *packed, int64_t packed_words);
ds_status ds_unpack_shift_weights_bits(const uint32_t *packed, int64_t rows, int64_t cols,
                                       int32_t bits, uint8_t *codes, int64_t codes_len);

/* LinearShift forward (Section 3, Y = W~ X + b with W~ = flip(2^P, S), Eq. 3):
 *     y[b][o] = bias[o] + sum_i term(x[b][i], code[o][i])    (mod 2^32)
 * x        device int32 [batch][in_features], fixed point with frac_bits F
 * w_packed device uint32 [out_features][ds_packed_row_words(in_features)]
 * bias     device int32 [out_features] with the same F, or NULL for none
 * y        device int32 [batch][out_features], written (not accumulated)
 * frac_bits in [0, 31]: the F of x, bias and y (validated, not used by the math)
 * flags    0, or DS_RELU: y = max(y, 0) after the sum (fused); with
 *          DS_CODE_BITS(b), w_packed holds b-bit codes (rows of
 *          ds_packed_row_words_bits(in_features, b) words)
 * stream   hipStream_t to enqueue on (NULL = default stream) */
ds_status ds_linear_shift(const int32_t *x, const uint32_t *w_packed, const int32_t *bias,
                          int32_t *y, int64_t batch, int64_t in_features, int64_t out_features,
                          int32_t frac_bits, uint32_t flags, void *stream);

/* ConvShift forward (Section 3, Y = W~ (*) X + b; Figure 1c), a 2-D
 * cross-correlation with zero padding, as an ordinary convolution layer:
 *     y[n][k][oh][ow] = bias[k] + sum_{c,r,s} term(x[n][c][ih][iw], code[k][c][r][s])
 *     ih = oh*stride_h - pad_h + r,  iw = ow*stride_w - pad_w + s
 * (positions outside the input contribute nothing), modulo 2^32.
 * x        device int32 [n][c][h][w] (NCHW), fixed point with frac_bits F
 * w_packed device uint32 [k][ds_packed_row_words(c*r*s)]; weight row k holds
 *          the codes in (c, r, s) order, s fastest
 * bias     device int32 [k] or NULL
 * y        device int32 [n][k][oh][ow],
 *          oh = (h + 2*pad_h - r)/stride_h + 1, ow = (w + 2*pad_w - s)/stride_w + 1
 * stride_* >= 1, pad_* >= 0; frac_bits, flags, stream as for ds_linear_shift. */
ds_status ds_conv2d_shift(const int32_t *x, const uint32_t *w_packed, const int32_t *bias,
                          int32_t *y, int64_t n, int64_t c, int64_t h, int64_t w,
                          int64_t k, int64_t r, int64_t s,
                          int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                          int32_t frac_bits, uint32_t flags, void *stream);

/* DeepShift-Q weight conversion (Section 3, Eqs. 4-5; range of Section 4):
 * float weights w -> packed codes of flip(2^p, s) with
 *     s = sign(w),  p = round(log2|w|) clipped to -max_shift .. 0.
 * round(log2|w|) is evaluated exactly (no float log): it has no ties for a
 * float w. w = +-0 and NaN give the zero weight (code 15); +-inf gives p = 0.
 * w        device float32 [rows][cols] (a weight row per output channel, as
 *          the compute entry points expect: cols = in_features or c*r*s)
 * max_shift in [0, 14]: 14 is the 5-bit format; smaller values give the
 *          shorter shift ranges of Section 4
 * w_packed device uint32 [rows][ds_packed_row_words(cols)], written
 *          ([rows][ds_packed_row_words_bits(cols, b)] with DS_CODE_BITS(b))
 * flags    0, or DS_CODE_BITS(b) to write b-bit codes, b in 2..5; then max_shift
 *          must be at most 2^(b-1) - 2; stream as for ds_linear_shift.
 * Errors: NULL pointer, rows/cols <= 0, max_shift out of range, output
 * overlapping the input, buffers that are not device allocations of the
 * required size, 2^31 or more elements. */
ds_status ds_quantize_shift_weights_q(const float *w, int64_t rows, int64_t cols,
                                      int32_t max_shift, uint32_t *w_packed,
                                      uint32_t flags, void *stream);

/* ds_quantize_shift_weights_q for `count` tensors in as few launches as
 * possible (one per 64 tensors): converting a whole network is then bound by
 * HBM bandwidth instead of per-launch latency. w, rows, cols and w_packed are
 * host arrays of `count` entries; w[i] and w_packed[i] are device pointers
 * with the layouts of ds_quantize_shift_weights_q. Every tensor is validated
 * before anything is launched (an error names the tensor), and no output may
 * overlap an input or another output. */
ds_status ds_quantize_shift_weights_q_many(int64_t count, const float *const *w,
                                           const int64_t *rows, const int64_t *cols,
                                           int32_t max_shift, uint32_t *const *w_packed,
                                           uint32_t flags, void *stream);

/* DeepShift-PS weight conversion (Section 3): from the shift parameters P and
 * the sign parameters S (device float32, both [rows][cols]):
 *     p = round(P) clipped to -max_shift .. 0,
 *     s = -1 if S <= -0.5, 0 if -0.5 < S < 0.5, +1 if S >= 0.5.
 * round() takes halves away from zero, the tie rule the sign thresholds state.
 * A NaN in P or S gives the zero weight. Other arguments and errors as for
 * ds_quantize_shift_weights_q. */
ds_status ds_quantize_shift_weights_ps(const float *p, const float *s, int64_t rows,
                                       int64_t cols, int32_t max_shift, uint32_t *w_packed,
                                       uint32_t flags, void *stream);

/* Fixed-point rounding of activations and bias (Section 4: 32-bit words with
 * 16 fractional bits):
 *     y[i] = round(x[i] * 2^frac_bits)
 * halves away from zero, saturated to [-2^31, 2^31 - 1]; NaN gives 0.
 * x device float32 [n]; y device int32 [n], written; y == x (in place) is
 * allowed, any other overlap is an error. frac_bits in [0, 31]; stream as for
 * ds_linear_shift. flags: 0, or DS_ACT_I16 / DS_ACT_I8 to write the lower
 * bit-width activations of Section 5: y is then int16 [n] (int8 [n]), saturated
 * to [-2^15, 2^15 - 1] ([-2^7, 2^7 - 1]), and must not overlap x. */
ds_status ds_to_fixed_point(const float *x, int64_t n, int32_t frac_bits, void *y,
                            uint32_t flags, void *stream);

/* ConvShift followed, in the same call, by what a ResNet block applies to a
 * convolution's output (batch normalisation, residual add, ReLU; fusing them
 * into the convolution is the optimisation Section 6 proposes). For each
 * output v = the ds_conv2d_shift result for channel k at flat index i:
 *     v = floor(v * mul[k] / 2^mul_shift) + add[k]     when mul != NULL
 *     v = v + residual[i]                              when residual != NULL
 *     v = max(v, 0)                                    when flags & DS_RELU
 * all in int32 with wrap-around (the product is formed in 64 bits). mul holds
 * a per-channel scale with mul_shift fractional bits (batch normalisation at
 * inference folds into it and add); add may be NULL (0) but needs mul.
 * mul, add: device int32 [k] or NULL; residual: device int32 with y's shape
 * [n][k][oh][ow] or NULL, and must not overlap y; mul_shift in [0, 31].
 * Other arguments and errors as for ds_conv2d_shift. */
ds_status ds_conv2d_shift_fused(const int32_t *x, const uint32_t *w_packed, const int32_t *bias,
                                const int32_t *mul, const int32_t *add, int32_t mul_shift,
                                const int32_t *residual, int32_t *y, int64_t n, int64_t c,
                                int64_t h, int64_t w, int64_t k, int64_t r, int64_t s,
                                int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                int32_t frac_bits, uint32_t flags, void *stream);

/* Max pooling of int32 x [n][c][h][w] into y [n][c][oh][ow] (oh, ow as for
 * ConvShift); window positions in the padding are ignored, so pad_h <= r/2 and
 * pad_w <= s/2 are required (every window then holds an input). The max pool
 * of the ResNet stem is r = s = 3, stride 2, pad 1. flags must be 0. */
ds_status ds_maxpool2d(const int32_t *x, int32_t *y, int64_t n, int64_t c, int64_t h, int64_t w,
                       int64_t r, int64_t s, int32_t stride_h, int32_t stride_w, int32_t pad_h,
                       int32_t pad_w, uint32_t flags, void *stream);

/* Global average pooling: y[n][c] = floor(sum over h*w of x[n][c] / (h*w)),
 * x device int32 [n][c][h][w], y device int32 [n][c]. flags must be 0. */
ds_status ds_avgpool2d_global(const int32_t *x, int32_t *y, int64_t n, int64_t c, int64_t h,
                              int64_t w, uint32_t flags, void *stream);

/* Input gradients (Section 3, the DeepShift backward pass): the gradient of
 * the loss with respect to an operator's input is the output gradient times
 * the same quantised weights -- transposed for LinearShift, and for ConvShift
 * the convolution of dY with the weights rotated by 180 degrees (the adjoint
 * of the forward convolution). In shift form every product of an output
 * gradient value g with a weight is term(g, code) as in the forward pass, so
 * the result is exact integer arithmetic like the forward one:
 *     dx[n][c][ih][iw] = sum over k, oh, ow, r, s with oh*stride_h - pad_h + r == ih
 *                        and ow*stride_w - pad_w + s == iw of
 *                        term(dy[n][k][oh][ow], code[k][c][r][s])      (mod 2^32)
 * dy and dx carry the same F (frac_bits, validated and not used by the math).
 *
 * ds_conv2d_shift_backward_data: the arguments describe the FORWARD layer
 * (n, c, h, w, k, r, s, stride, padding as for ds_conv2d_shift).
 * dy       device int32 [n][k][oh][ow] (oh, ow of the forward pass)
 * w_packed device uint32, the forward layer's packed weights [k][ds_packed_row_words(c*r*s)]
 * dx       device int32 [n][c][h][w], written (not accumulated); must not overlap dy or w_packed
 * flags    0, or DS_CODE_BITS(b) for b-bit packed codes; stream as for ds_linear_shift.
 * Device scratch (re-packed codes per stride phase, decoded weights) comes from
 * the library's stream-ordered pool, as for the forward operators.
 * Errors as for ds_conv2d_shift. */
ds_status ds_conv2d_shift_backward_data(const int32_t *dy, const uint32_t *w_packed, int32_t *dx,
                                        int64_t n, int64_t c, int64_t h, int64_t w, int64_t k,
                                        int64_t r, int64_t s, int32_t stride_h, int32_t stride_w,
                                        int32_t pad_h, int32_t pad_w, int32_t frac_bits,
                                        uint32_t flags, void *stream);

/* LinearShift input gradient: dx[b][i] = sum_o term(dy[b][o], code[o][i]) (mod 2^32).
 * dy device int32 [batch][out_features]; w_packed the forward layer's
 * [out_features][ds_packed_row_words(in_features)]; dx device int32
 * [batch][in_features], written. Other arguments and errors as above. */
ds_status ds_linear_shift_backward_data(const int32_t *dy, const uint32_t *w_packed, int32_t *dx,
                                        int64_t batch, int64_t in_features, int64_t out_features,
                                        int32_t frac_bits, uint32_t flags, void *stream);

/* Names, without launching anything, what ds_conv2d_shift_backward_data runs
 * for a forward layer of this shape: "direct" (one thread per dx element), or
 * "phases<P>" followed by each stride phase's window and kernel (a phase whose
 * rows or columns no tap reaches is "zero"). Arguments as for
 * ds_conv2d_shift_describe. For profiling and tests. */
ds_status ds_conv2d_shift_backward_data_describe(int64_t n, int64_t c, int64_t h, int64_t w,
                                                 int64_t k, int64_t r, int64_t s,
                                                 int32_t stride_h, int32_t stride_w,
                                                 int32_t pad_h, int32_t pad_w, char *buf,
                                                 int64_t len);

/* Multiplication-based comparison operators. Not part of DeepShift: they run
 * the same tiling as the shift operators with a 32-bit integer multiply in
 * place of the shift, so that the two inner loops can be timed side by side
 * (the paper compares its shift kernels with a multiplication-based kernel,
 * Section 6, GPU implementation). Weights are plain int32 [k][c*r*s]
 * (or [out][in]) on the device:
 *     y = bias + sum x * w    (products and sum modulo 2^32)
 * flags: 0, or DS_MUL_I24: each product is that of the low 24 bits of x and w,
 * each taken as a signed 24-bit value (one v_mad_i32_i24 per term), which equals
 * the int32 product while |x| < 2^23 and |w| < 2^23. */
#define DS_MUL_I24 4u
ds_status ds_conv2d_mul_i32(const int32_t *x, const int32_t *w, const int32_t *bias,
                            int32_t *y, int64_t n, int64_t c, int64_t h, int64_t w_,
                            int64_t k, int64_t r, int64_t s,
                            int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                            uint32_t flags, void *stream);
ds_status ds_linear_mul_i32(const int32_t *x, const int32_t *w, const int32_t *bias, int32_t *y,
                            int64_t batch, int64_t in_features, int64_t out_features,
                            uint32_t flags, void *stream);

/* Names, without launching anything, the kernel ds_conv2d_shift (or
 * ds_linear_shift, as a 1x1 convolution with h = w = 1) runs for a problem
 * of this shape on the current device, e.g. "tiled point tm8 cc8 splits1"
 * or "direct". Writes a NUL-terminated string of at most len bytes into buf.
 * Shape arguments are validated as for ds_conv2d_shift; no device memory is
 * touched. For profiling and tests. */
ds_status ds_conv2d_shift_describe(int64_t n, int64_t c, int64_t h, int64_t w, int64_t k,
                                   int64_t r, int64_t s, int32_t stride_h, int32_t stride_w,
                                   int32_t pad_h, int32_t pad_w, char *buf, int64_t len);

/* ---- Weight-specialised ConvShift (run-time code generation) --------------
 *
 * Section 6 of the paper proposes compiling the shift kernels for the weights
 * at hand. A plan is such a kernel: made once for fixed weights and a fixed
 * problem shape, it holds machine code in which every non-zero weight is one
 * integer add or subtract of a register that holds x >> shift, and zero
 * weights cost nothing. Run, it computes the same y as ds_conv2d_shift_fused
 * with the same bias, affine map, residual and ReLU, bit for bit:
 *     v = bias[k] + sum of term(x, code)                      (modulo 2^32)
 *     v = floor(v * mul[k] / 2^mul_shift) + add[k]            (when mul)
 *     v = v + residual[n][k][p]                               (DS_JIT_RESIDUAL)
 *     v = max(v, 0)                                           (DS_RELU)
 * Supported: any window up to 1023 columns wide, any stride and padding; a
 * LinearShift is the case h = w = r = s = 1. Windows over 3 x 3 read a
 * zero-padded copy of x, [n][c][xh][xw] with xh = (oh - 1) * stride_h + r and
 * xw = (ow - 1) * stride_w + s, that each run writes first into device memory
 * the plan holds (from create to destroy). A LinearShift of batch n >= 32 runs
 * on x^T: each run first transposes x into an int32 copy [c][n] the plan holds
 * (so that a load reads consecutive batch rows), the generated kernel writes
 * y^T [k][n] into a buffer the plan holds, and a last pass transposes it into
 * y (with the residual and the ReLU of a layer with a residual, and the whole
 * epilogue of a split reduction).
 *
 * ds_jit_conv_create: w_packed is HOST memory, [k][ds_packed_row_words(c*r*s)]
 * words as for ds_conv2d_shift (b-bit codes with DS_CODE_BITS(b) in flags); with
 * DS_ACT_I16 or DS_ACT_I8 in flags the plan's x is int16 or int8 (y and the
 * residual stay int32); bias, mul and add are HOST int32 [k] or NULL
 * (add needs mul; mul_shift in [0, 31] when mul is given). The plan copies
 * what it keeps; the caller's buffers may be freed on return. n, c, h, w and
 * the window fix the shape of every ds_jit_conv_run of the plan. splits: 0
 * chooses the split of the reduction over input channels (partial sums added
 * atomically into y); a positive value forces that many parts (at most c).
 * The plan's code is loaded on the current device with hipModuleLoadData and
 * lives until ds_jit_conv_destroy. Errors: as ds_conv2d_shift_fused for
 * arguments, DS_ERR_UNSUPPORTED for s > 1023 or a padded copy of 2^31 bytes or
 * more, DS_ERR_HIP when loading fails or device memory runs out. Making a plan
 * synchronises the device (module load, uploads).
 *
 * ds_jit_conv_run: x [n][c][h][w] (int32, or int16 / int8 for a plan made with
 * DS_ACT_I16 / DS_ACT_I8), residual and y [n][k][oh][ow] (int32), device
 * memory on the plan's device; residual must be non-NULL exactly when the
 * plan was made with DS_JIT_RESIDUAL. Asynchronous on `stream`. y must not
 * overlap x or residual. A plan may hold device scratch (the padded or
 * transposed copy of x; y^T; the partial sums of split strided phases of an
 * input-gradient plan), so runs
 * of one plan must not overlap in time: issue them on one stream, or order
 * them with events.
 *
 * ds_jit_conv_image: the code object ds_jit_conv_create would load, written
 * to host memory `image` of `capacity` bytes (*size = bytes needed;
 * DS_ERR_BUFFER_TOO_SMALL when capacity is short). Touches no device; for
 * inspection and tests.
 *
 * ds_jit_conv_query: size of the generated code in bytes, number of code
 * segments (up to 64 output channels x one part of the input channels each),
 * and the number of parts the reduction is split into. Any output may be NULL.
 *
 * ds_jit_conv_layout: how the plan's grid is laid out: output channels per
 * segment (16, 32 or 64), waves sharing each group of 64 pixels (the wave
 * split: 1, 2, 4, 8 or 16; each runs code of its own for a share of the
 * reduction), groups of 64 pixels per workgroup (1, 2 or 4; a workgroup has
 * groups x wave split <= 16 waves), pixel tiles (workgroups per segment), and
 * whether the plan runs a LinearShift on x^T (1) or not (0; its pixels are
 * then the batch rows of x, else the n pixels of x^T's one image). Each share's
 * code runs once per group of 64 pixels; segments x wave split distinct code
 * streams. For an input-gradient plan: its first kernel. Any output may be
 * NULL.
 *
 * Tuning overrides (ds_set_tuning, below) used when a plan is made (wave split,
 * loads in flight, register map, tile grouping, segment width) or run (block
 * order); for measurements only: DS_JIT_WSPLIT (1, 2, 4, 8 or 16 waves per 64
 * pixels), DS_JIT_TN (16, 32 or 64 output channels per segment), DS_JIT_PGROUPS
 * (1, 2 or 4 groups of 64 pixels per workgroup, at most 16 waves in all),
 * DS_JIT_SLOTS (loads in flight: 1-14, at most 8 in the 80-register code of
 * layers with one tap per element), DS_JIT_MAP (96: the 96-register code for
 * those layers too), DS_JIT_GROUP_TILES (tiles per group), DS_JIT_ORDER (0
 * grouped, 1 tile-major, 2 tile-major with each tile's workgroups on one XCD),
 * DS_JIT_TRANSPOSE (LinearShift plans on x^T: 0 never, 1 from batch 2).
 * The results do not depend on them. */
typedef struct ds_jit_conv ds_jit_conv;

ds_status ds_jit_conv_create(const uint32_t *w_packed, const int32_t *bias, const int32_t *mul,
                             const int32_t *add, int32_t mul_shift, int64_t n, int64_t c,
                             int64_t h, int64_t w, int64_t k, int64_t r, int64_t s,
                             int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                             uint32_t flags, int32_t splits, ds_jit_conv **plan);
ds_status ds_jit_conv_run(const ds_jit_conv *plan, const void *x, const int32_t *residual,
                          int32_t *y, void *stream);
ds_status ds_jit_conv_destroy(ds_jit_conv *plan);
ds_status ds_jit_conv_image(const uint32_t *w_packed, const int32_t *bias, const int32_t *mul,
                            const int32_t *add, int32_t mul_shift, int64_t n, int64_t c,
                            int64_t h, int64_t w, int64_t k, int64_t r, int64_t s,
                            int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                            uint32_t flags, int32_t splits, void *image, int64_t capacity,
                            int64_t *size);
ds_status ds_jit_conv_query(const ds_jit_conv *plan, int64_t *code_bytes, int32_t *segments,
                            int32_t *splits);
ds_status ds_jit_conv_layout(const ds_jit_conv *plan, int32_t *channels, int32_t *wsplit,
                             int32_t *pixel_groups, int32_t *pixel_tiles, int32_t *transposed);

/* A plan for the input gradient of a ConvShift layer (the result of
 * ds_conv2d_shift_backward_data, bit for bit), with the weights baked into
 * the code as for ds_jit_conv_create. The arguments describe the FORWARD layer;
 * w_packed is HOST memory (b-bit codes with DS_CODE_BITS(b), the only flag).
 * The plan splits dx into the stride phases of the layer, each a generated
 * kernel writing its own rows and columns of dx; ds_jit_conv_run(plan, dy,
 * NULL, dx, stream) then takes dy [n][k][oh][ow] and writes all of dx
 * [n][c][h][w] (residual must be NULL). A LinearShift is the case
 * h = w = r = s = 1; from batch 32 its plan runs on dy^T as a forward
 * LinearShift plan runs on x^T. Phases with windows over 3 x 3 read a padded
 * copy of dy as forward plans do. DS_ERR_UNSUPPORTED when a phase is wider than 1023
 * columns. ds_jit_conv_query reports the code of all phases. Other errors as
 * for ds_jit_conv_create. */
ds_status ds_jit_conv_backward_data_create(const uint32_t *w_packed, int64_t n, int64_t c,
                                           int64_t h, int64_t w, int64_t k, int64_t r, int64_t s,
                                           int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                           int32_t pad_w, uint32_t flags, int32_t splits,
                                           ds_jit_conv **plan);

/* Multiplication plans: the multiplication-based comparison operator (not
 * DeepShift; Section 6 times the shift kernels against a multiplication-based
 * kernel) in the tiling of the weight-specialised plans above, so that the two
 * can be timed side by side: the same template kernel, register map, wave
 * split, split-K and block order, with each non-zero weight one
 * v_mad_i32_i24 (the weight an inline constant or an s_mov_b32 literal) in
 * place of the shift plans' add or subtract. Zero weights cost nothing.
 *     y = bias + sum over the window of x * w      (modulo 2^32)
 * where each product is that of the low 24 bits of x and w taken as signed
 * 24-bit values: the int32 product while |x| < 2^23 and |w| < 2^23, as
 * ds_conv2d_mul_i32 with DS_MUL_I24.
 * w HOST int32 [k][c*r*s]; bias HOST int32 [k] or NULL; flags 0 or DS_RELU;
 * other arguments, errors and the run / destroy / query calls as for
 * ds_jit_conv_create. ds_jit_conv_mul_image writes the code object as
 * ds_jit_conv_image does. */
ds_status ds_jit_conv_mul_create(const int32_t *w, const int32_t *bias, int64_t n, int64_t c,
                                 int64_t h, int64_t w_, int64_t k, int64_t r, int64_t s,
                                 int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                 uint32_t flags, int32_t splits, ds_jit_conv **plan);
ds_status ds_jit_conv_mul_image(const int32_t *w, const int32_t *bias, int64_t n, int64_t c,
                                int64_t h, int64_t w_, int64_t k, int64_t r, int64_t s,
                                int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                uint32_t flags, int32_t splits, void *image, int64_t capacity,
                                int64_t *size);

/* ---- ConvShift that allocates nothing ------------------------------------
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.
 * ds_conv2d_shift_noalloc computes exactly what ds_conv2d_shift computes (same
 * arguments, layouts, flags and errors; a LinearShift is the case
 * h = w = r = s = 1 with x [batch][in] as [batch][in][1][1]) and calls no
 * hipMalloc, hipMallocAsync, hipFree or other allocating routine. Its scratch
 * is one array of DS_NOALLOC_SCRATCH_BYTES per GPU, placed in the library's
 * code object and held from the library's first use on that GPU until the
 * process ends. A problem whose scratch would exceed it fails with
 * DS_ERR_UNSUPPORTED before anything is launched; ds_conv2d_shift_noalloc_
 * scratch_bytes gives a shape's need (-1 for an invalid shape; 0 for shapes
 * on the one-thread-per-output kernel). Every call on a GPU uses that GPU's one
 * array: calls on one stream are ordered, but calls that overlap in time on
 * one GPU (several streams, several host threads) race on it and must be
 * serialised by the caller. */
#define DS_NOALLOC_SCRATCH_BYTES (32u << 20)
ds_status ds_conv2d_shift_noalloc(const int32_t *x, const uint32_t *w_packed, const int32_t *bias,
                                  int32_t *y, int64_t n, int64_t c, int64_t h, int64_t w,
                                  int64_t k, int64_t r, int64_t s,
                                  int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                  int32_t frac_bits, uint32_t flags, void *stream);
int64_t ds_conv2d_shift_noalloc_scratch_bytes(int64_t n, int64_t c, int64_t h, int64_t w,
                                              int64_t k, int64_t r, int64_t s, int32_t stride_h,
                                              int32_t stride_w, int32_t pad_h, int32_t pad_w);

/* Tuning overrides, for tests and measurements: they change which kernel
 * variant, wave split, block order or load depth the library uses, never a
 * result. Knobs: "DS_FORCE_VARIANT" (0: the one-thread-per-output kernel for
 * ds_conv2d_shift and the input gradients; 8: the tiled kernel with 8 pixels
 * per lane where one exists), "DS_ROWS_BATCH" (1, 2, 4 or 8 batch rows per
 * workgroup of the kernel that runs a LinearShift below 256 rows) and the plan
 * knobs listed with ds_jit_conv_create.
 * Each starts from the environment variable of the same name, read once when
 * the library is loaded (unset: -1, the library's own choice); no entry point
 * reads the environment afterwards. value < 0 resets a knob to -1. Errors:
 * NULL pointer, unknown name (DS_ERR_INVALID_ARG). Thread-safe; a change is
 * seen by calls and plans made after it. */
ds_status ds_set_tuning(const char *name, int32_t value);
ds_status ds_get_tuning(const char *name, int32_t *value);

/* Static text for a status code. */
const char *ds_status_string(ds_status status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char *ds_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* DEEPSHIFT_H */
