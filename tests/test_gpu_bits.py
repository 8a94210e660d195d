"""GPU parity with weights packed in fewer bits (DS_CODE_BITS, Section 5's
shorter shift ranges): every entry point that reads packed weights, given b-bit
codes (b = 2, 3, 4), matches the oracle run on the same weights in the 5-bit
form, bit for bit: ConvShift (tiled and one-thread-per-output kernels, split and
unsplit), the fused epilogue, LinearShift, both input gradients, and
weight-specialised plans.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
BITS = [2, 3, 4]


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def codes_for(rng, shape, bits, zero_frac=0.15):
    ones = (1 << (bits - 1)) - 1
    shift = rng.integers(0, ones, shape) if ones > 0 else np.zeros(shape, np.int64)
    shift[rng.random(shape) < zero_frac] = 15
    return (rng.integers(0, 2, shape) << 4 | shift).astype(np.uint8)


def packed(codes, bits):
    return to_dev(ops.pack_shift_weights(codes, bits=bits).view(np.int32))


CONV = [(2, 13, 9, 11, 37, 3, 1, 1), (3, 20, 15, 15, 33, 1, 2, 0), (1, 300, 6, 6, 3, 3, 1, 1),
        (4, 64, 20, 20, 128, 3, 2, 1)]


@pytest.mark.parametrize("bits", BITS)
@pytest.mark.parametrize("direct", [False, True], ids=["tiled", "direct"])
def test_conv_matches_oracle(bits, direct, knob):
    if direct:
        knob("DS_FORCE_VARIANT", 0)
    for shape in CONV:
        n, c, h, w, k, r, st, pd = shape
        rng = np.random.default_rng(zlib.crc32(repr((shape, bits)).encode()))
        x = rng.integers(-(2 ** 31), 2 ** 31, (n, c, h, w), dtype=np.int64).astype(np.int32)
        codes = codes_for(rng, (k, c * r * r), bits)
        bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
        y = ops.conv2d_shift(to_dev(x), packed(codes, bits), to_dev(bias), r, st, pd, code_bits=bits)
        np.testing.assert_array_equal(y.cpu().numpy(),
                                      oracle.conv2d_shift(x, codes, bias, r=r, stride=st, pad=pd))


@pytest.mark.parametrize("bits", BITS)
def test_fused_and_linear_match_oracle(bits):
    rng = np.random.default_rng(bits)
    n, c, h, k = 2, 24, 11, 70
    x = rng.integers(-(2 ** 22), 2 ** 22, (n, c, h, h)).astype(np.int32)
    codes = codes_for(rng, (k, c * 9), bits)
    mul = rng.integers(-(2 ** 17), 2 ** 17, k).astype(np.int32)
    add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    res = rng.integers(-(2 ** 24), 2 ** 24, (n, k, h, h)).astype(np.int32)
    y = ops.conv2d_shift_fused(to_dev(x), packed(codes, bits), None, 3, 1, 1, mul=to_dev(mul),
                               add=to_dev(add), mul_shift=16, residual=to_dev(res), relu=True,
                               code_bits=bits)
    want = oracle.epilogue(oracle.conv2d_shift(x, codes, None, r=3, stride=1, pad=1), mul, add, 16,
                           residual=res, relu=True)
    np.testing.assert_array_equal(y.cpu().numpy(), want)
    xl = rng.integers(-(2 ** 31), 2 ** 31, (33, 300), dtype=np.int64).astype(np.int32)
    cl = codes_for(rng, (70, 300), bits)
    bl = rng.integers(-(2 ** 16), 2 ** 16, 70).astype(np.int32)
    yl = ops.linear_shift(to_dev(xl), packed(cl, bits), to_dev(bl), code_bits=bits)
    np.testing.assert_array_equal(yl.cpu().numpy(), oracle.linear_shift(xl, cl, bl))


@pytest.mark.parametrize("bits", BITS)
def test_input_gradients_match_oracle(bits):
    rng = np.random.default_rng(10 + bits)
    for (n, c, h, w, k, r, st, pd) in CONV:
        oh, ow = (h + 2 * pd - r) // st + 1, (w + 2 * pd - r) // st + 1
        dy = rng.integers(-(2 ** 31), 2 ** 31, (n, k, oh, ow), dtype=np.int64).astype(np.int32)
        codes = codes_for(rng, (k, c * r * r), bits)
        dx = ops.conv2d_shift_backward_data(to_dev(dy), packed(codes, bits), (n, c, h, w), r, st, pd,
                                            code_bits=bits)
        np.testing.assert_array_equal(dx.cpu().numpy(), oracle.conv2d_shift_backward_data(
            dy, codes, (n, c, h, w), r=r, stride=st, pad=pd))
    dyl = rng.integers(-(2 ** 31), 2 ** 31, (16, 70), dtype=np.int64).astype(np.int32)
    cl = codes_for(rng, (70, 300), bits)
    dxl = ops.linear_shift_backward_data(to_dev(dyl), packed(cl, bits), 300, code_bits=bits)
    np.testing.assert_array_equal(dxl.cpu().numpy(), oracle.linear_shift_backward_data(dyl, cl))


@pytest.mark.parametrize("bits", BITS)
def test_weight_specialised_plan_matches_oracle(bits):
    rng = np.random.default_rng(20 + bits)
    n, c, h, w, k = 3, 13, 9, 11, 70
    x = rng.integers(-(2 ** 31), 2 ** 31, (n, c, h, w), dtype=np.int64).astype(np.int32)
    codes = codes_for(rng, (k, c * 9), bits)
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    plan = ops.JitConv(ops.pack_shift_weights(codes, bits=bits), x.shape, 3, 1, 1, bias=bias,
                       code_bits=bits)
    y = plan(to_dev(x)).cpu().numpy()
    plan.close()
    np.testing.assert_array_equal(y, oracle.conv2d_shift(x, codes, bias, r=3, stride=1, pad=1))


@pytest.mark.parametrize("bits", BITS)
def test_converters_write_b_bit_codes(bits):
    """DeepShift-Q and DeepShift-PS straight into b-bit codes: the words unpack (oracle)
    to the oracle's codes with the b-bit shift range."""
    from paper_1905_13298_amd import workloads as W
    max_shift = (1 << (bits - 1)) - 2
    shapes = [(64, 27), (70, 576), (3, 1)]
    ws = [W.gen_float_weights(r, c, seed=300 + i) for i, (r, c) in enumerate(shapes)]
    outs = ops.quantize_shift_weights_q_many([to_dev(w) for w in ws], max_shift=max_shift,
                                             code_bits=bits)
    for w, o, (r, c) in zip(ws, outs, shapes):
        words = o.cpu().numpy().view(np.uint32)
        np.testing.assert_array_equal(oracle.unpack_codes_bits(words, c, bits),
                                      oracle.quantize_q(w, max_shift).reshape(r, c))
        np.testing.assert_array_equal(words, oracle.pack_codes_bits(oracle.quantize_q(w, max_shift), bits))
    p, s = W.gen_ps_params(50, 99, seed=bits, p_range=(-6.0, 1.0))
    got = ops.quantize_shift_weights_ps(to_dev(p), to_dev(s), max_shift=max_shift, code_bits=bits)
    np.testing.assert_array_equal(got.cpu().numpy().view(np.uint32),
                                  oracle.pack_codes_bits(oracle.quantize_ps(p, s, max_shift), bits))
