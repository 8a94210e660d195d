"""GPU parity on seeded random problems with random layouts.

Each case draws a ConvShift (with or without the fused epilogue: per-channel
affine, residual, ReLU), a LinearShift, or a ConvShift input gradient, with
random shapes, strides, padding, signs, zero-weight fractions, weight codes of
2 to 5 bits, plan inputs of 32, 16 or 8 bits, forced plan
layouts (segment width, wave split, pixel groups, block order and its tile
groups, loads in flight, register map, split-K parts, x^T or x for LinearShift,
batch rows per workgroup of the small-batch kernel),
and compares the runtime-weights call and the weight-specialised plan with the
oracle bit for bit. The layouts are the ones the planner can be forced into
for measurements; every one of them must give the oracle's output.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops
from paper_1905_13298_amd.workloads import random_codes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
KNOBS = ("DS_JIT_TN", "DS_JIT_WSPLIT", "DS_JIT_PGROUPS", "DS_JIT_ORDER", "DS_JIT_TRANSPOSE",
         "DS_ROWS_BATCH", "DS_JIT_SLOTS", "DS_JIT_MAP", "DS_JIT_GROUP_TILES")
CASES = 400


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


DT = {32: np.int32, 16: np.int16, 8: np.int8}


def draw_codes(rng, shape):
    """Codes in the 5-bit form whose shifts fit b bits (b = 2..5), and b."""
    bits = int(rng.choice([5, 5, 5, 4, 3, 2]))
    zero_frac = float(rng.choice([0.0, 0.1, 0.3, 0.9]))
    if bits == 5:
        return random_codes(rng, shape, zero_frac=zero_frac), bits
    ones = (1 << (bits - 1)) - 1
    shift = rng.integers(0, ones, shape) if ones > 0 else np.zeros(shape, np.int64)
    shift[rng.random(shape) < zero_frac] = 15
    return (rng.integers(0, 2, shape) << 4 | shift).astype(np.uint8), bits


def draw_x(rng, shape, signed, act_bits):
    if act_bits == 32:
        return rng.integers(-(2 ** 24) if signed else 0, 2 ** 24, shape).astype(np.int32)
    info = np.iinfo(DT[act_bits])
    return rng.integers(info.min if signed else 0, info.max, shape, endpoint=True).astype(DT[act_bits])


def draw_knobs(rng, knob):
    v = {k: -1 for k in KNOBS}
    if rng.random() < 0.6:
        v["DS_JIT_TN"] = int(rng.choice([-1, 16, 32, 64]))
        ws, pg = int(rng.choice([-1, 1, 2, 4, 8, 16])), int(rng.choice([-1, 1, 2, 4]))
        if ws > 0 and pg > 0 and ws * pg > 16:
            pg = -1
        if ws == 16 and pg != 1:
            pg = -1
        v["DS_JIT_WSPLIT"], v["DS_JIT_PGROUPS"] = ws, pg
        v["DS_JIT_ORDER"] = int(rng.choice([-1, 0, 1, 2]))
    v["DS_JIT_TRANSPOSE"] = int(rng.choice([-1, -1, 0, 1]))
    v["DS_ROWS_BATCH"] = int(rng.choice([-1, -1, 1, 2, 4, 8]))
    v["DS_JIT_SLOTS"] = int(rng.choice([-1, -1, 1, 2, 3, 5, 8, 14]))
    v["DS_JIT_MAP"] = int(rng.choice([-1, -1, -1, 96]))
    v["DS_JIT_GROUP_TILES"] = int(rng.choice([-1, -1, 1, 2, 7, 64]))
    for k, x in v.items():
        knob(k, x)
    return v


def assert_equal(name, got, want, info):
    bad = np.flatnonzero(got.ravel() != want.ravel())
    assert bad.size == 0, f"{name} {info}: {bad.size} of {want.size} outputs differ, first at {bad[:5]}"


def linear_case(rng, info):
    b, c, k = int(rng.integers(1, 300)), int(rng.integers(1, 700)), int(rng.integers(1, 500))
    signed = bool(rng.random() < 0.5)
    act_bits = int(rng.choice([32, 32, 16, 8]))
    x = draw_x(rng, (b, c), signed, act_bits)
    codes, bits = draw_codes(rng, (k, c))
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32) if rng.random() < 0.7 else None
    relu = bool(rng.random() < 0.3)
    splits = int(rng.choice([0, 0, 1, 2, 3]))
    info += ("linear", b, c, k, signed, act_bits, bits, relu, bias is not None, splits)
    say("case", info)
    x32 = x.astype(np.int32)
    want = oracle.linear_shift(x32, codes, bias)
    if relu:
        want = np.maximum(want, 0)
    wp = ops.pack_shift_weights(codes, bits=bits)
    y = ops.linear_shift(to_dev(x32), to_dev(wp.view(np.int32)), to_dev(bias), relu=relu,
                         code_bits=bits)
    assert_equal("runtime", y.cpu().numpy(), want, info)
    plan = ops.JitConv(wp, (b, c, 1, 1), 1, 1, 0, bias=bias, relu=relu, splits=splits,
                       code_bits=bits, act_bits=act_bits)
    try:
        y = plan(to_dev(x).view(b, c, 1, 1)).cpu().numpy().reshape(b, k)
        assert_equal("plan", y, want, info + (plan.channels, plan.wsplit, plan.pixel_groups,
                                              plan.splits, plan.transposed))
    finally:
        plan.close()


def conv_shape(rng):
    while True:
        n, c, k = int(rng.integers(1, 7)), int(rng.integers(1, 160)), int(rng.integers(1, 160))
        r, s = int(rng.integers(1, 8)), int(rng.integers(1, 8))
        st, pd = int(rng.integers(1, 4)), int(rng.integers(0, 4))
        h, w = int(rng.integers(1, 37)), int(rng.integers(1, 37))
        if h + 2 * pd >= r and w + 2 * pd >= s and n * c * k * r * s * h * w <= 2e8:
            return n, c, h, w, k, r, s, st, pd


def gradient_case(rng, info):
    n, c, h, w, k, r, s, st, pd = conv_shape(rng)
    codes, bits = draw_codes(rng, (k, c * r * s))
    oh, ow = (h + 2 * pd - r) // st + 1, (w + 2 * pd - s) // st + 1
    dy = rng.integers(-(2 ** 24), 2 ** 24, (n, k, oh, ow)).astype(np.int32)
    splits = int(rng.choice([0, 0, 1, 2]))
    info += ("gradient", n, c, h, w, k, r, s, st, pd, bits, splits)
    say("case", info)
    want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, w), r=r, s=s, stride=st, pad=pd)
    wp = ops.pack_shift_weights(codes, bits=bits)
    y = ops.conv2d_shift_backward_data(to_dev(dy), to_dev(wp.view(np.int32)), (n, c, h, w), (r, s),
                                       st, pd, code_bits=bits)
    assert_equal("runtime", y.cpu().numpy(), want, info)
    plan = ops.JitConvBackwardData(wp, (n, c, h, w), (r, s), st, pd, splits=splits, code_bits=bits)
    try:
        assert_equal("plan", plan(to_dev(dy)).cpu().numpy(), want,
                     info + (plan.channels, plan.wsplit, plan.pixel_groups, plan.splits))
    finally:
        plan.close()


def conv_case(rng, info):
    n, c, h, w, k, r, s, st, pd = conv_shape(rng)
    signed = bool(rng.random() < 0.5)
    act_bits = int(rng.choice([32, 32, 16, 8]))
    x = draw_x(rng, (n, c, h, w), signed, act_bits)
    codes, bits = draw_codes(rng, (k, c * r * s))
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32) if rng.random() < 0.5 else None
    oh, ow = (h + 2 * pd - r) // st + 1, (w + 2 * pd - s) // st + 1
    ep = bool(rng.random() < 0.5)
    mul = rng.integers(1, 2 ** 17, k).astype(np.int32) if ep and rng.random() < 0.7 else None
    add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32) if mul is not None else None
    res = rng.integers(-(2 ** 24), 2 ** 24, (n, k, oh, ow)).astype(np.int32) \
        if ep and rng.random() < 0.5 else None
    relu = bool(ep and rng.random() < 0.5)
    splits = int(rng.choice([0, 0, 1, 2, 3]))
    info += ("conv", n, c, h, w, k, r, s, st, pd, signed, act_bits, bits, bias is not None,
             mul is not None, res is not None, relu, splits)
    say("case", info)
    x32 = x.astype(np.int32)
    want = oracle.conv2d_shift(x32, codes, bias, r=r, s=s, stride=st, pad=pd)
    if ep:
        want = oracle.epilogue(want, mul, add, 16, res, relu)
    wp = ops.pack_shift_weights(codes, bits=bits)
    xd, wd = to_dev(x), to_dev(wp.view(np.int32))
    # The runtime-weights calls read int32 inputs: the narrow values widened, whose
    # terms equal the narrow plan's (an arithmetic shift of a sign-extended value).
    if ep:
        y = ops.conv2d_shift_fused(to_dev(x32), wd, to_dev(bias), (r, s), st, pd, to_dev(mul), to_dev(add),
                                   16, to_dev(res), relu, code_bits=bits)
    else:
        y = ops.conv2d_shift(to_dev(x32), wd, to_dev(bias), (r, s), st, pd, code_bits=bits)
    assert_equal("runtime", y.cpu().numpy(), want, info)
    plan = ops.JitConv(wp, x.shape, (r, s), st, pd, bias=bias, mul=mul, add=add,
                       residual=res is not None, relu=relu, splits=splits, code_bits=bits,
                       act_bits=act_bits)
    try:
        assert_equal("plan", plan(xd, residual=to_dev(res)).cpu().numpy(), want,
                     info + (plan.channels, plan.wsplit, plan.pixel_groups, plan.splits))
    finally:
        plan.close()


@pytest.mark.parametrize("seed", [1905, 13298])
def test_random_problems_in_random_layouts(seed, knob):
    rng = np.random.default_rng(seed)
    for i in range(CASES):
        info = (seed, i, draw_knobs(rng, knob))
        kind = rng.choice(["conv", "conv", "conv", "linear", "gradient"])
        {"conv": conv_case, "linear": linear_case, "gradient": gradient_case}[kind](rng, info)
