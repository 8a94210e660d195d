"""Pins for the oracle's layers around the shift convolutions (chained inference).

* the epilogue's affine map against numpy's int64 arithmetic right shift (a
  floor) on the exact product, its wrap-around against Python integers, ReLU
  against ``numpy.maximum``, and the order affine -> residual -> ReLU by
  composing those library routines;
* max pooling against ``torch.nn.functional.max_pool2d`` in float64 (int32
  values are exact in float64; torch pads with -inf, i.e. ignores padding);
* global average pooling against ``numpy.floor_divide`` of int64 sums, and a
  constant input that must come back unchanged.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

I32 = np.iinfo(np.int32)


def wrap(v):
    return ((np.asarray(v, dtype=object) + 2 ** 31) % 2 ** 32 - 2 ** 31).astype(np.int64)


@pytest.mark.parametrize("mul_shift", [0, 5, 16, 31])
def test_epilogue_affine_matches_numpy_shift(mul_shift):
    rng = np.random.default_rng(mul_shift)
    N, K, P = 3, 7, 11
    y = rng.integers(I32.min, I32.max, (N, K, P), dtype=np.int64).astype(np.int32)
    y[0, 0, :4] = [0, -1, 1, I32.min]
    mul = rng.integers(-(2 ** 20), 2 ** 20, K).astype(np.int32)
    add = rng.integers(I32.min, I32.max, K, dtype=np.int64).astype(np.int32)
    got = oracle.epilogue(y, mul, add, mul_shift)
    prod = y.astype(np.int64) * mul[None, :, None].astype(np.int64)
    want = wrap(np.right_shift(prod, mul_shift).astype(object) + add[None, :, None].astype(object))
    np.testing.assert_array_equal(got.astype(np.int64), want)


def test_epilogue_residual_then_relu_order():
    rng = np.random.default_rng(1)
    y = rng.integers(-(2 ** 20), 2 ** 20, (2, 5, 3, 4)).astype(np.int32)
    res = rng.integers(-(2 ** 20), 2 ** 20, y.shape).astype(np.int32)
    mul = rng.integers(1, 2 ** 17, 5).astype(np.int32)
    add = rng.integers(-(2 ** 16), 2 ** 16, 5).astype(np.int32)
    got = oracle.epilogue(y, mul, add, 16, residual=res, relu=True)
    aff = np.right_shift(y.astype(np.int64) * mul[None, :, None, None], 16) + add[None, :, None, None]
    want = np.maximum(aff + res, 0)
    np.testing.assert_array_equal(got.astype(np.int64), want)
    # residual and ReLU alone; an identity affine (mul = 2^s, add = 0) changes nothing
    np.testing.assert_array_equal(oracle.epilogue(y, residual=res), y.astype(np.int64) + res)
    np.testing.assert_array_equal(oracle.epilogue(y, relu=True), np.maximum(y, 0))
    ident = np.full(5, 1 << 16, np.int32)
    np.testing.assert_array_equal(oracle.epilogue(y, ident, None, 16), y)


def test_epilogue_wraps_residual_sum():
    y = np.array([[[I32.max, I32.min, -5]]], np.int32)
    res = np.array([[[1, -1, 5]]], np.int32)
    np.testing.assert_array_equal(oracle.epilogue(y, residual=res), [[[I32.min, I32.max, 0]]])


@pytest.mark.parametrize("shape", [(2, 3, 9, 9, 3, 2, 1), (1, 4, 8, 7, 3, 2, 1), (2, 2, 6, 6, 2, 2, 0),
                                   (1, 1, 5, 5, 3, 1, 1), (1, 2, 112, 112, 3, 2, 1)])
def test_maxpool_matches_torch(shape):
    n, c, h, w, r, st, pd = shape
    rng = np.random.default_rng(h * w + r)
    x = rng.integers(I32.min, I32.max, (n, c, h, w), dtype=np.int64).astype(np.int32)
    x[..., :2, :2] = -(2 ** 31)   # all-negative corners: padding must not win
    got = oracle.maxpool2d(x, r=r, stride=st, pad=pd)
    want = F.max_pool2d(torch.from_numpy(x.astype(np.float64)), r, st, pd).numpy()
    np.testing.assert_array_equal(got.astype(np.float64), want)


def test_avgpool_global_matches_numpy():
    rng = np.random.default_rng(3)
    x = rng.integers(I32.min, I32.max, (3, 5, 7, 7), dtype=np.int64).astype(np.int32)
    got = oracle.avgpool_global(x)
    want = np.floor_divide(x.astype(np.int64).reshape(3, 5, -1).sum(-1), 49)
    np.testing.assert_array_equal(got.astype(np.int64), want)
    const = np.full((2, 3, 7, 7), -12345, np.int32)
    np.testing.assert_array_equal(oracle.avgpool_global(const), np.full((2, 3), -12345))
