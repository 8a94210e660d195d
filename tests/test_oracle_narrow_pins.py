"""Pins of the oracle on the lower bit-width activations (Section 5): 16-bit
activations in 3.13 fixed point and 8-bit ones in 3.5.

The oracle sign-extends int16 / int8 activations to int32 and applies the int32
operator. These tests pin that against definitions written out independently:

* brute force with Python integers on tiny shapes -- every term is
  floor(x / 2^s) on the narrow value itself, negated after the shift, summed
  exactly and wrapped once -- for every code and the extreme narrow values;
* the closed form: 16-bit inputs that are multiples of 2^14 make every shift
  exact, so the result equals a float64 convolution with weights sign * 2^-s
  (the paper's float emulation);
* the narrow fixed-point rounding against exact rational arithmetic (halves away
  from zero, saturation at the type's range, NaN -> 0).
"""
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

BITS = [(16, 13, np.int16), (8, 5, np.int8)]


def wrap(v):
    return ((v + 2 ** 31) % 2 ** 32) - 2 ** 31


def brute_conv(x, codes, bias, r, s, stride, pad):
    N, C, H, W = x.shape
    K = codes.shape[0]
    OH, OW = (H + 2 * pad - r) // stride + 1, (W + 2 * pad - s) // stride + 1
    y = np.zeros((N, K, OH, OW), np.int64)
    for n in range(N):
        for k in range(K):
            for oh in range(OH):
                for ow in range(OW):
                    acc = int(bias[k]) if bias is not None else 0
                    for c in range(C):
                        for i in range(r):
                            for j in range(s):
                                ih, iw = oh * stride - pad + i, ow * stride - pad + j
                                if not (0 <= ih < H and 0 <= iw < W):
                                    continue
                                code = int(codes[k, (c * r + i) * s + j])
                                sh, neg = code & 15, code >> 4
                                if sh == 15:
                                    continue
                                t = int(x[n, c, ih, iw]) // (1 << sh)   # floor on the narrow value
                                acc += -t if neg else t
                    y[n, k, oh, ow] = wrap(acc)
    return y


@pytest.mark.parametrize("bits,frac,dt", BITS, ids=["i16", "i8"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_narrow_brute_force(bits, frac, dt, seed):
    rng = np.random.default_rng([bits, seed])
    info = np.iinfo(dt)
    n, c, h, w, k = 2, 3, 5, 6, 32
    r, s, stride, pad = [(3, 3, 1, 1), (2, 3, 2, 1), (1, 1, 1, 0)][seed]
    x = rng.integers(info.min, info.max, (n, c, h, w), endpoint=True).astype(dt)
    x.flat[:4] = [info.min, info.max, -1, 1]
    # every code in every row and column position
    codes = ((rng.permutation(k)[:, None] + 5 * np.arange(c * r * s)[None, :]) % 32).astype(np.uint8)
    bias = rng.integers(-(1 << frac), 1 << frac, k).astype(np.int32)
    want = brute_conv(x, codes, bias, r, s, stride, pad)
    got = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=stride, pad=pad)
    np.testing.assert_array_equal(got.astype(np.int64), want)
    # LinearShift on narrow rows
    xl = rng.integers(info.min, info.max, (4, 40), endpoint=True).astype(dt)
    cl = (np.arange(40)[None, :] * 7 + np.arange(9)[:, None] * 3).astype(np.uint8) % 32
    want_l = brute_conv(xl.reshape(4, 40, 1, 1), cl, None, 1, 1, 1, 0).reshape(4, 9)
    np.testing.assert_array_equal(oracle.linear_shift(xl, cl, None).astype(np.int64), want_l)


def test_int16_closed_form_at_3_13():
    """Multiples of 2^14 in int16 (-2^15, -2^14, 0, 2^14) shift exactly by 0..14."""
    rng = np.random.default_rng(13)
    x = (rng.integers(-2, 2, (2, 4, 7, 7)) * (1 << 14)).astype(np.int16)
    codes = rng.integers(0, 32, (6, 4 * 9)).astype(np.uint8)
    got = oracle.conv2d_shift(x, codes, None, r=3, stride=1, pad=1).astype(np.float64)
    sh = (codes & 15).astype(np.int64)
    wf = np.where(sh == 15, 0.0, np.ldexp(1.0, -np.minimum(sh, 14)))
    wf = np.where((codes >> 4) & 1, -wf, wf).reshape(6, 4, 3, 3)
    ref = F.conv2d(torch.from_numpy(x.astype(np.float64)), torch.from_numpy(wf), padding=1).numpy()
    np.testing.assert_array_equal(got, ref)


def exact_round(v, frac, bits):
    if v != v:
        return 0
    lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    if v in (float("inf"), float("-inf")):
        return hi if v > 0 else lo
    q = Fraction(v) * (1 << frac)
    fl = q.numerator // q.denominator
    rem = q - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and q > 0):
        r_ = fl + 1
    else:
        r_ = fl
    return max(lo, min(hi, r_))


@pytest.mark.parametrize("bits,frac,dt", BITS, ids=["i16", "i8"])
def test_narrow_fixed_point_rounding(bits, frac, dt):
    rng = np.random.default_rng(bits)
    scale = 2.0 ** (bits - 1 - frac)                       # the format's range
    v = (rng.standard_normal(4000) * scale).astype(np.float32)
    ties = ((np.arange(-40, 40) + 0.5) / (1 << frac)).astype(np.float32)
    special = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, scale, -scale, 3 * scale, -3 * scale,
                        np.float32(scale) - np.float32(2.0 ** -frac)], np.float32)
    x = np.concatenate([v, ties, special]).astype(np.float32)
    got = oracle.to_fixed_narrow(x, frac, bits)
    assert got.dtype == dt
    want = np.array([exact_round(float(t), frac, bits) for t in x], dtype=np.int64)
    np.testing.assert_array_equal(got.astype(np.int64), want)
