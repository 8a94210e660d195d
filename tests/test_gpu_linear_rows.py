"""GPU parity of the small-batch LinearShift kernel (lanes own output channels;
batches below 256 rows), bit for bit against the oracle: ragged batch, input and
output sizes, the widest int32 inputs, every code, 2-5-bit codes, the fused
epilogue and ReLU, the multiplication comparison operators in the same tiling,
and the entry point that allocates nothing (the kernel needs no scratch)."""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import _native, ops

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def draw(seed, b, c, k, bits=5):
    rng = np.random.default_rng(seed)
    x = rng.integers(-(2 ** 31), 2 ** 31, (b, c), dtype=np.int64).astype(np.int32)
    x.flat[: min(x.size, 4)] = [-(2 ** 31), 2 ** 31 - 1, -1, 0][: min(x.size, 4)]
    top = (1 << bits) - 1
    raw = rng.integers(0, top + 1, (k, c))
    # b-bit codes as the canonical 5-bit form (sign bit on top, all-ones shift = zero)
    sh_bits = bits - 1
    sh = raw & ((1 << sh_bits) - 1)
    sign = raw >> sh_bits
    codes = ((sign << 4) | np.where(sh == (1 << sh_bits) - 1, 15, sh)).astype(np.uint8)
    bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
    return x, codes, bias, rng


SHAPES = [
    # batch, in, out
    (1, 1, 1), (1, 5, 3), (1, 6, 64), (1, 7, 65), (2, 300, 130), (3, 97, 63), (5, 4100, 70),
    (8, 256, 128), (9, 512, 1000), (17, 61, 129), (31, 1000, 17), (100, 2048, 200), (255, 37, 300),
]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{b}x{c}to{k}" for b, c, k in SHAPES])
def test_small_batch_linear_matches_oracle(shape):
    b, c, k = shape
    x, codes, bias, _ = draw(zlib.crc32(repr(shape).encode()), b, c, k)
    assert ops.describe_conv2d(b, c, 1, 1, k, 1) == "rows"
    wt = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    y = ops.linear_shift(to_dev(x), wt, to_dev(bias)).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.linear_shift(x, codes, bias))
    # no bias, ReLU
    y = ops.linear_shift(to_dev(x), wt, None, relu=True).cpu().numpy()
    np.testing.assert_array_equal(y, np.maximum(oracle.linear_shift(x, codes, None), 0))


# batch, in, out: a long reduction that splits over workgroups, a short one that does not
FORCED = [(13, 4100, 70), (11, 333, 129)]


@pytest.mark.parametrize("rows", [1, 2, 4, 8])
@pytest.mark.parametrize("shape", FORCED, ids=[f"{b}x{c}to{k}" for b, c, k in FORCED])
def test_small_batch_rows_per_workgroup_match_oracle(shape, rows):
    """Every batch-rows tiling (the batch not a multiple of it) gives the oracle's
    result, with the reduction split over workgroups or not."""
    b, c, k = shape
    x, codes, bias, _ = draw(zlib.crc32(repr((shape, rows)).encode()), b, c, k)
    wt = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    with ops.tuning("DS_ROWS_BATCH", rows):
        y = ops.linear_shift(to_dev(x), wt, to_dev(bias)).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.linear_shift(x, codes, bias))


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_small_batch_linear_code_widths(bits):
    b, c, k = 5, 203, 77
    x, codes, bias, _ = draw(bits, b, c, k, bits)
    wp = ops.pack_shift_weights(codes, bits=bits)   # canonical codes, packed in `bits` bits
    y = ops.linear_shift(to_dev(x), to_dev(wp.view(np.int32)), to_dev(bias), code_bits=bits).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.linear_shift(x, codes, bias))


def test_small_batch_fused_epilogue_matches_oracle():
    b, c, k = 6, 333, 90
    x, codes, bias, rng = draw(11, b, c, k)
    x = (x >> 12).astype(np.int32)
    mul = rng.integers(-(2 ** 17), 2 ** 17, k).astype(np.int32)
    add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    res = rng.integers(-(2 ** 24), 2 ** 24, (b, k, 1, 1)).astype(np.int32)
    y = ops.conv2d_shift_fused(to_dev(x.reshape(b, c, 1, 1)), to_dev(ops.pack_shift_weights(codes).view(np.int32)),
                               to_dev(bias), 1, mul=to_dev(mul), add=to_dev(add), mul_shift=16,
                               residual=to_dev(res), relu=True).cpu().numpy()
    conv = oracle.conv2d_shift(x.reshape(b, c, 1, 1), codes, bias, r=1)
    np.testing.assert_array_equal(y, oracle.epilogue(conv, mul, add, 16, residual=res, relu=True))


@pytest.mark.parametrize("mul24", [False, True], ids=["i32", "i24"])
def test_small_batch_multiplication_comparison(mul24):
    b, c, k = 7, 300, 130
    rng = np.random.default_rng(5 + mul24)
    x = rng.integers(-(2 ** 31), 2 ** 31, (b, c), dtype=np.int64).astype(np.int32)
    w = rng.integers(-(2 ** 31), 2 ** 31, (k, c), dtype=np.int64).astype(np.int32)
    y = ops.linear_mul_i32(to_dev(x), to_dev(w), mul24=mul24).cpu().numpy()
    if mul24:
        want = oracle.conv2d_mul24(x.reshape(b, c, 1, 1), w, None, r=1).reshape(b, k)
    else:
        want = oracle.conv2d_mul(x.reshape(b, c, 1, 1), w, None, r=1).reshape(b, k)
    np.testing.assert_array_equal(y, want)


def test_small_batch_noalloc_needs_no_scratch():
    b, c, k = 3, 4096, 4096
    assert _native.lib().ds_conv2d_shift_noalloc_scratch_bytes(b, c, 1, 1, k, 1, 1, 1, 1, 0, 0) == 0
    x, codes, bias, _ = draw(21, b, c, k)
    xt, wt, bt = to_dev(x), to_dev(ops.pack_shift_weights(codes).view(np.int32)), to_dev(bias)
    y = torch.empty((b, k), dtype=torch.int32, device=DEV)
    st = _native.lib().ds_conv2d_shift_noalloc(xt.data_ptr(), wt.data_ptr(), bt.data_ptr(), y.data_ptr(),
                                               b, c, 1, 1, k, 1, 1, 1, 1, 0, 0, 16, 0, None)
    assert st == 0
    np.testing.assert_array_equal(y.cpu().numpy(), oracle.linear_shift(x, codes, bias))
