/*
 * Oracle for the DeepShift shift operators -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU implementation of what LinearShift and ConvShift compute
 * at inference time. Only the tests, the smoke check and the benchmark's CPU
 * baseline use it; the product library never calls it and shares no code
 * with it.
 *
 * What is computed (DeepShift, Section 3, Eqs. 1-3; Figure 1a; Section 4):
 *   Each weight is flip(2^p, s) with p an integer power and s a ternary sign
 *   (Eq. 3). Multiplying a fixed-point activation x by 2^p is a bitwise shift
 *   (Eq. 1); the powers used are 0 .. -14, so every shift is a right shift by
 *   -p. The sign flip (Eq. 2) negates, keeps or zeroes the shifted value, and
 *   the products are summed as in an ordinary linear layer or convolution,
 *   plus a bias (Section 3, Y = W X + b and Y = W (*) X + b).
 *
 * Readings where the paper is silent (each one is also listed in the design
 * notes of this project):
 *   - A right shift of a negative x rounds toward minus infinity (an
 *     arithmetic shift): term = floor(x * 2^p). The paper equates the shift
 *     with the multiplication, which is exact only when the low bits are 0.
 *   - The shift is applied first and the sign flip second: -(floor(x*2^p)).
 *   - Weight code (uint8): bit 4 = sign (1 means negate), bits 0-3 = shift
 *     code c; c in 0..14 means p = -c; c = 15 means a zero weight whatever
 *     the sign bit (the ternary zero of Eq. 2 within the 5-bit budget of
 *     Section 4).
 *   - Sums are formed exactly (int64 here) and wrapped once to int32
 *     (two's complement, modulo 2^32).
 *   - Bias is optional (NULL) and is added once per output.
 *   - Packed layout: six 5-bit codes per uint32 word, code j of the word in
 *     bits [5j, 5j+5), bits 30-31 zero; each weight row starts a new word and
 *     its last word is filled with code 15.
 *
 * Input gradients (Section 3, backward pass): the same terms applied to the
 * output gradient and summed over the forward connections (the adjoint), see
 * oracle_conv2d_shift_backward_data.
 *
 * The floor is computed by integer division, not by the shift operator, so
 * the oracle does not rely on how C shifts negative numbers.
 *
 * Parity status: every function here is pinned by the CPU test suite
 * (brute force with exact rationals, the closed form against a float64
 * library convolution on inputs divisible by 2^15, a library arithmetic
 * shift, the one-sided rounding bound, zero-code and sign-flip invariants,
 * and hand-derived packed words). The converter functions at the end are
 * pinned against numpy's float64 log2/round, exact rational rounding, the
 * paper's second form of the ternary sign (sign of round(S)), the
 * nearest-power property, and hand-derived examples. The layers for chained
 * inference at the end are pinned against numpy's int64 arithmetic shift and
 * floor division and torch's max pooling. The input gradients are pinned
 * against torch's float64 conv2d input gradient on inputs divisible by 2^15
 * (closed form), the adjoint identity <W x, g> = <x, W^T g> with exact
 * integers, a brute-force gather loop in Python, the transposed-codes forward
 * pass for LinearShift and for stride-1 convolutions, and the one-sided
 * rounding bound.
 */
#include <stdint.h>
#include <limits.h>
#include <stddef.h>
#include <math.h>
#include <stdlib.h>

/* floor(x / 2^c) for 0 <= c <= 14, by integer division (Eq. 1, reading: floor). */
static int64_t floor_div_pow2(int64_t x, int c)
{
    int64_t d = (int64_t)1 << c;
    int64_t q = x / d;            /* C division truncates toward zero */
    if (x % d != 0 && x < 0)
        q -= 1;                   /* move truncation down to the floor */
    return q;
}

/* One weight applied to one activation: flip(floor(x * 2^p), s) (Eqs. 1-3). */
int64_t oracle_term(int32_t x, uint8_t code)
{
    int shift = code & 15;
    int negative = (code >> 4) & 1;
    if (shift == 15)
        return 0;                 /* zero weight (s = 0 in Eq. 2) */
    int64_t t = floor_div_pow2((int64_t)x, shift);
    return negative ? -t : t;
}

/* Two's-complement wrap of an exact sum to int32 (modulo 2^32). */
static int32_t wrap32(int64_t v)
{
    uint32_t u = (uint32_t)(uint64_t)v;
    return (int32_t)u;            /* gcc: modulo conversion */
}

/* LinearShift, Y = W~ X + b (Section 3): x [batch][in], codes [out][in],
 * bias [out] or NULL, y [batch][out]. */
void oracle_linear_shift(const int32_t *x, const uint8_t *codes, const int32_t *bias,
                         int32_t *y, int64_t batch, int64_t in, int64_t out)
{
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t o = 0; o < out; ++o) {
            int64_t acc = bias ? (int64_t)bias[o] : 0;
            for (int64_t i = 0; i < in; ++i)
                acc += oracle_term(x[b * in + i], codes[o * in + i]);
            y[b * out + o] = wrap32(acc);
        }
    }
}

/* ConvShift output element (n, k, oh, ow): Y = W~ (*) X + b (Section 3).
 * x [N][C][H][W], codes [K][C][R][S] (flattened rows of C*R*S), zero padding. */
static int32_t conv_point(const int32_t *x, const uint8_t *codes, const int32_t *bias,
                          int64_t C, int64_t H, int64_t W, int64_t R, int64_t S,
                          int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                          int64_t n, int64_t k, int64_t oh, int64_t ow)
{
    int64_t acc = bias ? (int64_t)bias[k] : 0;
    for (int64_t c = 0; c < C; ++c)
        for (int64_t r = 0; r < R; ++r)
            for (int64_t s = 0; s < S; ++s) {
                int64_t ih = oh * sh - ph + r;
                int64_t iw = ow * sw - pw + s;
                if (ih < 0 || ih >= H || iw < 0 || iw >= W)
                    continue;     /* zero padding contributes nothing */
                int32_t xv = x[((n * C + c) * H + ih) * W + iw];
                uint8_t code = codes[((k * C + c) * R + r) * S + s];
                acc += oracle_term(xv, code);
            }
    return wrap32(acc);
}

static int64_t out_dim(int64_t in, int64_t pad, int64_t k, int64_t stride)
{
    return (in + 2 * pad - k) / stride + 1;
}

void oracle_conv2d_shift(const int32_t *x, const uint8_t *codes, const int32_t *bias,
                         int32_t *y, int64_t N, int64_t C, int64_t H, int64_t W,
                         int64_t K, int64_t R, int64_t S, int64_t sh, int64_t sw,
                         int64_t ph, int64_t pw)
{
    int64_t OH = out_dim(H, ph, R, sh), OW = out_dim(W, pw, S, sw);
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            for (int64_t oh = 0; oh < OH; ++oh)
                for (int64_t ow = 0; ow < OW; ++ow)
                    y[((n * K + k) * OH + oh) * OW + ow] =
                        conv_point(x, codes, bias, C, H, W, R, S, sh, sw, ph, pw,
                                   n, k, oh, ow);
}

/* Selected outputs of a convolution: idx holds flattened indices into y
 * [N][K][OH][OW]; out[i] receives y[idx[i]]. */
void oracle_conv2d_shift_points(const int32_t *x, const uint8_t *codes, const int32_t *bias,
                                int64_t N, int64_t C, int64_t H, int64_t W, int64_t K,
                                int64_t R, int64_t S, int64_t sh, int64_t sw, int64_t ph,
                                int64_t pw, const int64_t *idx, int64_t npts, int32_t *out)
{
    int64_t OH = out_dim(H, ph, R, sh), OW = out_dim(W, pw, S, sw);
    (void)N;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < npts; ++i) {
        int64_t t = idx[i];
        int64_t ow = t % OW; t /= OW;
        int64_t oh = t % OH; t /= OH;
        int64_t k = t % K;   t /= K;
        out[i] = conv_point(x, codes, bias, C, H, W, R, S, sh, sw, ph, pw, t, k, oh, ow);
    }
}

/* Selected outputs of a linear layer: idx into y [batch][out]. */
void oracle_linear_shift_points(const int32_t *x, const uint8_t *codes, const int32_t *bias,
                                int64_t batch, int64_t in, int64_t out_features,
                                const int64_t *idx, int64_t npts, int32_t *out)
{
    (void)batch;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < npts; ++i) {
        int64_t b = idx[i] / out_features, o = idx[i] % out_features;
        int64_t acc = bias ? (int64_t)bias[o] : 0;
        for (int64_t j = 0; j < in; ++j)
            acc += oracle_term(x[b * in + j], codes[o * in + j]);
        out[i] = wrap32(acc);
    }
}

/* ---- Input gradients (the data half of the backward pass) ------------------
 *
 * Section 3 (DeepShift-Q backward pass, with its footnote): the gradient of the
 * loss with respect to the operator input is the output gradient multiplied by
 * the same quantised weights: dX = dY W~ for LinearShift (W~ transposed, in
 * the footnote's words), and the convolution of dY with W~ rotated by 180
 * degrees for ConvShift, i.e. the adjoint of the forward convolution. In shift
 * form each product of an output-gradient value g (fixed point) with a weight
 * is the same term(g, code) as in the forward pass (floor shift, then the
 * sign); sums are exact and wrapped once.
 *
 * The definition used here is the adjoint written as a scatter: every forward
 * connection (output (n, k, oh, ow), tap (c, r, s), input (ih, iw)) sends
 * term(dy[n][k][oh][ow], code[k][c][r][s]) back to dx[n][c][ih][iw]. */

/* dx [batch][in] = sum_o term(dy[b][o], code[o][i]); dy [batch][out]. */
void oracle_linear_shift_backward_data(const int32_t *dy, const uint8_t *codes, int32_t *dx,
                                       int64_t batch, int64_t in, int64_t out)
{
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t i = 0; i < in; ++i) {
            int64_t acc = 0;
            for (int64_t o = 0; o < out; ++o)
                acc += oracle_term(dy[b * out + o], codes[o * in + i]);
            dx[b * in + i] = wrap32(acc);
        }
}

/* dx [N][C][H][W] from dy [N][K][OH][OW] (OH, OW of the forward pass). */
void oracle_conv2d_shift_backward_data(const int32_t *dy, const uint8_t *codes, int32_t *dx,
                                       int64_t N, int64_t C, int64_t H, int64_t W, int64_t K,
                                       int64_t R, int64_t S, int64_t sh, int64_t sw,
                                       int64_t ph, int64_t pw)
{
    int64_t OH = out_dim(H, ph, R, sh), OW = out_dim(W, pw, S, sw);
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c) {
            /* each (n, c) plane of dx is written by this iteration only */
            int64_t *acc = (int64_t *)calloc((size_t)(H * W), sizeof(int64_t));
            for (int64_t k = 0; k < K; ++k)
                for (int64_t oh = 0; oh < OH; ++oh)
                    for (int64_t ow = 0; ow < OW; ++ow) {
                        int32_t g = dy[((n * K + k) * OH + oh) * OW + ow];
                        for (int64_t r = 0; r < R; ++r)
                            for (int64_t s = 0; s < S; ++s) {
                                int64_t ih = oh * sh - ph + r, iw = ow * sw - pw + s;
                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)
                                    continue;  /* the forward pass read padding here */
                                acc[ih * W + iw] +=
                                    oracle_term(g, codes[((k * C + c) * R + r) * S + s]);
                            }
                    }
            for (int64_t i = 0; i < H * W; ++i)
                dx[(n * C + c) * H * W + i] = wrap32(acc[i]);
            free(acc);
        }
}

/* Selected elements dx.flat[idx[i]] of the input gradient, each gathered on its
 * own: the taps (r, s) and outputs (oh, ow) with oh*sh - ph + r == ih and
 * ow*sw - pw + s == iw. */
void oracle_conv2d_shift_backward_data_points(const int32_t *dy, const uint8_t *codes,
                                              int64_t N, int64_t C, int64_t H, int64_t W,
                                              int64_t K, int64_t R, int64_t S, int64_t sh,
                                              int64_t sw, int64_t ph, int64_t pw,
                                              const int64_t *idx, int64_t npts, int32_t *out)
{
    int64_t OH = out_dim(H, ph, R, sh), OW = out_dim(W, pw, S, sw);
    (void)N;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < npts; ++i) {
        int64_t t = idx[i];
        int64_t iw = t % W; t /= W;
        int64_t ih = t % H; t /= H;
        int64_t c = t % C;  t /= C;
        int64_t n = t;
        int64_t acc = 0;
        for (int64_t k = 0; k < K; ++k)
            for (int64_t r = 0; r < R; ++r) {
                int64_t a = ih + ph - r;           /* = oh * sh */
                if (a < 0 || a % sh != 0 || a / sh >= OH)
                    continue;
                for (int64_t s = 0; s < S; ++s) {
                    int64_t b = iw + pw - s;       /* = ow * sw */
                    if (b < 0 || b % sw != 0 || b / sw >= OW)
                        continue;
                    acc += oracle_term(dy[((n * K + k) * OH + a / sh) * OW + b / sw],
                                       codes[((k * C + c) * R + r) * S + s]);
                }
            }
        out[i] = wrap32(acc);
    }
}

/* Multiplication-based comparison operator: y = wrap32(b + sum x * w) with
 * int32 weights, products and sums exact. Same layouts as the shift ops. */
void oracle_conv2d_mul(const int32_t *x, const int32_t *wts, const int32_t *bias, int32_t *y,
                       int64_t N, int64_t C, int64_t H, int64_t W, int64_t K, int64_t R,
                       int64_t S, int64_t sh, int64_t sw, int64_t ph, int64_t pw)
{
    int64_t OH = out_dim(H, ph, R, sh), OW = out_dim(W, pw, S, sw);
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            for (int64_t oh = 0; oh < OH; ++oh)
                for (int64_t ow = 0; ow < OW; ++ow) {
                    int64_t acc = bias ? (int64_t)bias[k] : 0;
                    for (int64_t c = 0; c < C; ++c)
                        for (int64_t r = 0; r < R; ++r)
                            for (int64_t s = 0; s < S; ++s) {
                                int64_t ih = oh * sh - ph + r, iw = ow * sw - pw + s;
                                if (ih < 0 || ih >= H || iw < 0 || iw >= W)
                                    continue;
                                acc += (int64_t)x[((n * C + c) * H + ih) * W + iw] *
                                       (int64_t)wts[((k * C + c) * R + r) * S + s];
                            }
                    y[((n * K + k) * OH + oh) * OW + ow] = wrap32(acc);
                }
}

/* Packed layout (reading: see header): rows x cols codes -> rows x ceil(cols/6)
 * words. Codes must be < 32. */
void oracle_pack_codes(const uint8_t *codes, int64_t rows, int64_t cols, uint32_t *packed)
{
    int64_t wpr = (cols + 5) / 6;
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t w = 0; w < wpr; ++w) {
            uint32_t word = 0;
            for (int64_t j = 0; j < 6; ++j) {
                int64_t col = w * 6 + j;
                uint32_t code = col < cols ? codes[r * cols + col] : 15u;
                word |= (code & 31u) << (5 * j);
            }
            packed[r * wpr + w] = word;
        }
}

void oracle_unpack_codes(const uint32_t *packed, int64_t rows, int64_t cols, uint8_t *codes)
{
    int64_t wpr = (cols + 5) / 6;
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t col = 0; col < cols; ++col)
            codes[r * cols + col] =
                (uint8_t)((packed[r * wpr + col / 6] >> (5 * (col % 6))) & 31u);
}

/* Weight codes in fewer bits (Section 5 trains with shift values limited to
 * shorter ranges). Reading: a b-bit code (b = 2..5) keeps the sign in its top
 * bit and the shift code in the b-1 bits below it; the all-ones shift code is
 * the zero weight, so shifts run 0 .. -(2^(b-1) - 2) (b = 5 gives the 0 .. -14
 * and code 15 of the 5-bit format). floor(32 / b) codes fill a word from bit 0
 * up, rows start on a new word, the last word is padded with the zero weight.
 * Codes are given and returned in the 5-bit form (sign << 4 | shift code).
 * Returns -1 (and writes nothing) when a code's shift does not fit b bits. */
int oracle_pack_codes_bits(const uint8_t *codes, int64_t rows, int64_t cols, int bits,
                           uint32_t *packed)
{
    int64_t per = 32 / bits, wpr = (cols + per - 1) / per;
    uint32_t ones = (1u << (bits - 1)) - 1u;
    for (int64_t i = 0; i < rows * cols; ++i) {
        uint32_t shift = codes[i] & 15u;
        if (shift != 15u && shift >= ones)
            return -1;
    }
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t w = 0; w < wpr; ++w) {
            uint32_t word = 0;
            for (int64_t j = 0; j < per; ++j) {
                int64_t col = w * per + j;
                uint32_t field = ones, sign = 0;
                if (col < cols) {
                    uint32_t code = codes[r * cols + col];
                    sign = (code >> 4) & 1u;
                    field = (code & 15u) == 15u ? ones : (code & 15u);
                }
                word |= ((sign << (bits - 1)) | field) << (bits * j);
            }
            packed[r * wpr + w] = word;
        }
    return 0;
}

void oracle_unpack_codes_bits(const uint32_t *packed, int64_t rows, int64_t cols, int bits,
                              uint8_t *codes)
{
    int64_t per = 32 / bits, wpr = (cols + per - 1) / per;
    uint32_t ones = (1u << (bits - 1)) - 1u;
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t col = 0; col < cols; ++col) {
            uint32_t raw = (packed[r * wpr + col / per] >> (bits * (col % per))) & ((1u << bits) - 1u);
            uint32_t field = raw & ones, sign = raw >> (bits - 1);
            codes[r * cols + col] = (uint8_t)((sign << 4) | (field == ones ? 15u : field));
        }
}

/* ------------------------------------------------------------------------
 * Float -> weight code converter and fixed-point conversion.
 *
 * DeepShift-Q (Section 3, Eqs. 4-5): s = sign(w), p = round(log2|w|).
 * DeepShift-PS (Section 3): p = round(P), s = -1 if S <= -0.5, 0 if
 * -0.5 < S < 0.5, +1 if S >= 0.5.
 * Both clip p to the supported range -max_shift .. 0 (Section 4; 14 for the
 * 5-bit format). Inputs and bias are rounded to fixed point with F fractional
 * bits (Section 4, 16.16).
 *
 * Readings where the paper is silent:
 *   - The only tie rule the paper states is the one for the sign (+-0.5 go to
 *     +-1, i.e. halves away from zero); round(P) and the fixed-point rounding
 *     use the same rule. round(log2|w|) has no ties for a float w (log2|w| =
 *     p + 1/2 would need |w| = 2^p * sqrt(2), which is irrational).
 *   - w = +-0 has sign 0, i.e. the zero weight. A NaN (w, P or S) also gives
 *     the zero weight; w = +-inf gives p = 0 after clipping.
 *   - Fixed point saturates to the int32 range; NaN gives 0.
 */

/* round(log2|w|) for finite w != 0, evaluated exactly: with p = floor(log2|w|),
 * |w| lies in [2^p, 2^(p+1)) and rounds up iff |w| >= 2^(p + 1/2), i.e. iff
 * w^2 >= 2^(2p+1). Both sides are exact in double for a float w. */
static int round_log2_abs(float w)
{
    int e;
    (void)frexp(fabs((double)w), &e);        /* |w| = m * 2^e with m in [0.5, 1) */
    const int p = e - 1;                     /* floor(log2|w|) */
    const double w2 = (double)w * (double)w;
    return (w2 >= ldexp(1.0, 2 * p + 1)) ? p + 1 : p;
}

/* Code of flip(2^p, s) with p clipped to -max_shift .. 0; s = 0 -> code 15. */
static uint8_t code_of(int p, int s, int max_shift)
{
    if (s == 0) return 15;
    if (p > 0) p = 0;
    if (p < -max_shift) p = -max_shift;
    return (uint8_t)((s < 0 ? 16 : 0) | (-p));
}

/* DeepShift-Q codes of n float weights (any layout; one code per weight). */
void oracle_quantize_q(const float *w, int64_t n, int max_shift, uint8_t *codes)
{
    for (int64_t i = 0; i < n; ++i) {
        const float v = w[i];
        int s = (v > 0.0f) - (v < 0.0f);     /* sign(w); NaN -> 0 */
        int p = (s == 0 || isinf(v)) ? 0 : round_log2_abs(v);
        codes[i] = code_of(p, s, max_shift);
    }
}

/* DeepShift-PS codes from the shift parameters P and sign parameters S. */
void oracle_quantize_ps(const float *P, const float *S, int64_t n, int max_shift, uint8_t *codes)
{
    for (int64_t i = 0; i < n; ++i) {
        const float sv = S[i];
        int s = sv <= -0.5f ? -1 : (sv >= 0.5f ? 1 : 0);   /* NaN -> 0 */
        const double r = round((double)P[i]);              /* halves away from zero */
        if (isnan(r)) s = 0;
        int p = (r > 0.0) ? 0 : (r < -64.0 ? -64 : (int)r);
        codes[i] = code_of(p, s, max_shift);
    }
}

/* Fixed point with F fractional bits: round(x * 2^F), halves away from zero,
 * saturated to int32; NaN -> 0. */
void oracle_to_fixed(const float *x, int64_t n, int frac_bits, int32_t *out)
{
    for (int64_t i = 0; i < n; ++i) {
        const double v = (double)x[i];
        if (isnan(v)) { out[i] = 0; continue; }
        const double t = round(ldexp(v, frac_bits));
        if (t >= 2147483647.0) out[i] = 2147483647;
        else if (t <= -2147483648.0) out[i] = -2147483647 - 1;
        else out[i] = (int32_t)t;
    }
}

/* ------------------------------------------------------------------------
 * Layers around the shift convolutions, for chained inference: the network
 * the paper times in Section 6 (ResNet-18) keeps batch normalisation, max and
 * average pooling and residual connections next to its shift convolutions.
 * Here they act on the same int32 fixed-point values (any F).
 *
 * Readings where the paper is silent:
 *   - Batch normalisation at inference is a per-channel affine map, applied
 *     as v * mul[k] / 2^mul_shift + add[k] with the division floored (the
 *     rounding of the shift operators) and the result wrapped to int32.
 *   - The residual is added after the affine map and before ReLU (the order of
 *     a ResNet basic block), wrapping to int32; ReLU is max(v, 0).
 *   - Max pooling ignores window positions in the padding.
 *   - Global average pooling floors the division of the sum by H * W.
 */

/* floor(v / 2^s) for 0 <= s <= 62, by integer division. */
static int64_t floor_div_pow2_64(int64_t v, int s)
{
    int64_t d = (int64_t)1 << s;
    int64_t q = v / d;
    if (v % d != 0 && v < 0)
        q -= 1;
    return q;
}

/* In place on y [N][K][P] (P = OH * OW): affine (when mul is not NULL; add may
 * be NULL), then + residual[i] (when not NULL), then ReLU (when relu != 0). */
void oracle_epilogue(int32_t *y, int64_t N, int64_t K, int64_t P, const int32_t *mul,
                     const int32_t *add, int mul_shift, const int32_t *residual, int relu)
{
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            for (int64_t p = 0; p < P; ++p) {
                int64_t i = (n * K + k) * P + p;
                int64_t v = y[i];
                if (mul) {
                    v = floor_div_pow2_64(v * (int64_t)mul[k], mul_shift);
                    v = wrap32(v + (add ? (int64_t)add[k] : 0));
                }
                if (residual)
                    v = wrap32(v + (int64_t)residual[i]);
                if (relu && v < 0)
                    v = 0;
                y[i] = (int32_t)v;
            }
}

/* Max pooling, x [N][C][H][W] -> y [N][C][OH][OW]; padding positions are ignored
 * (the caller keeps pad <= R/2, S/2 so that every window holds an input). */
void oracle_maxpool2d(const int32_t *x, int32_t *y, int64_t N, int64_t C, int64_t H, int64_t W,
                      int64_t R, int64_t S, int64_t sh, int64_t sw, int64_t ph, int64_t pw)
{
    int64_t OH = out_dim(H, ph, R, sh), OW = out_dim(W, pw, S, sw);
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c)
            for (int64_t oh = 0; oh < OH; ++oh)
                for (int64_t ow = 0; ow < OW; ++ow) {
                    int64_t best = INT64_MIN;
                    for (int64_t r = 0; r < R; ++r)
                        for (int64_t s = 0; s < S; ++s) {
                            int64_t ih = oh * sh - ph + r, iw = ow * sw - pw + s;
                            if (ih < 0 || ih >= H || iw < 0 || iw >= W)
                                continue;
                            int64_t v = x[((n * C + c) * H + ih) * W + iw];
                            if (v > best)
                                best = v;
                        }
                    y[((n * C + c) * OH + oh) * OW + ow] = (int32_t)best;
                }
}

/* Global average pooling, x [N][C][HW] -> y [N][C]: floor(sum / HW). */
void oracle_avgpool_global(const int32_t *x, int32_t *y, int64_t N, int64_t C, int64_t HW)
{
    for (int64_t i = 0; i < N * C; ++i) {
        int64_t sum = 0;
        for (int64_t p = 0; p < HW; ++p)
            sum += x[i * HW + p];
        int64_t q = sum / HW;
        if (sum % HW != 0 && sum < 0)
            q -= 1;
        y[i] = (int32_t)q;
    }
}
