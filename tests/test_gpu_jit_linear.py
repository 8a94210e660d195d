"""GPU parity of weight-specialised LinearShift plans on x^T (the default from
batch 32, forced here from batch 2 with DS_JIT_TRANSPOSE = 1), which run their
kernel on an int32 copy of x^T (loads of 64 consecutive batch rows of one input
channel) and write y^T, transposed back into y by a last pass that adds the
residual and applies the ReLU of a layer with one.
Bit for bit against the oracle: ragged batches around the 64-row tiles,
every epilogue part whole and split over parts of the reduction, forced
segment widths, wave splits and pixel groups, int16 / int8 activations, the
multiplication plans (comparison operator), and two runs of one plan."""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.fixture(autouse=True)
def transposed(knob):
    knob("DS_JIT_TRANSPOSE", 1)


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def draw(seed, n, c, k, lim=2 ** 31):
    rng = np.random.default_rng(seed)
    sign = rng.integers(0, 2, (k, c))
    shift = rng.integers(0, 16, (k, c))
    codes = (sign << 4 | shift).astype(np.uint8)
    x = rng.integers(-lim, lim, (n, c), dtype=np.int64).astype(np.int32)
    bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
    return codes, x, bias, rng


SHAPES = [(2, 7, 3), (33, 40, 17), (64, 64, 64), (65, 130, 70), (130, 300, 129), (256, 512, 200),
          (300, 97, 65)]


@pytest.mark.parametrize("splits", [1, 0, 3])
@pytest.mark.parametrize("shape", SHAPES, ids=[f"{n}x{c}to{k}" for n, c, k in SHAPES])
def test_transposed_linear_plans_match_oracle(shape, splits):
    n, c, k = shape
    codes, x, bias, _ = draw(zlib.crc32(repr((shape, splits)).encode()), n, c, k)
    say(f"jit linear {shape} splits={splits}")
    plan = ops.JitConv(ops.pack_shift_weights(codes), (n, c, 1, 1), 1, bias=bias, splits=splits)
    y = plan(to_dev(x.reshape(n, c, 1, 1))).cpu().numpy().reshape(n, k)
    plan.close()
    np.testing.assert_array_equal(y, oracle.linear_shift(x, codes, bias))


@pytest.mark.parametrize("splits", [1, 2])
@pytest.mark.parametrize("parts", ["mul_add", "residual", "residual_relu", "all", "relu"])
def test_transposed_linear_epilogue_matches_oracle(parts, splits):
    n, c, k = 77, 150, 90
    codes, x, bias, rng = draw(zlib.crc32(parts.encode()) + splits, n, c, k, lim=2 ** 18)
    mul = add = res = None
    if "mul" in parts or parts == "all":
        mul = rng.integers(-(2 ** 17), 2 ** 17, k).astype(np.int32)
    if "add" in parts or parts == "all":
        add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    if "residual" in parts or parts == "all":
        res = rng.integers(-(2 ** 24), 2 ** 24, (n, k, 1, 1)).astype(np.int32)
    relu = "relu" in parts or parts == "all"
    say(f"jit linear epilogue {parts} splits={splits}")
    plan = ops.JitConv(ops.pack_shift_weights(codes), (n, c, 1, 1), 1, bias=bias, mul=mul, add=add,
                       mul_shift=16, residual=res is not None, relu=relu, splits=splits)
    y = plan(to_dev(x.reshape(n, c, 1, 1)), residual=to_dev(res)).cpu().numpy()
    plan.close()
    conv = oracle.conv2d_shift(x.reshape(n, c, 1, 1), codes, bias, r=1)
    np.testing.assert_array_equal(y, oracle.epilogue(conv, mul, add, 16, residual=res, relu=relu))


LAYOUTS = [(64, 1, 4), (64, 4, 4), (64, 16, 1), (32, 8, 2), (16, 4, 4), (16, 2, 1)]


@pytest.mark.parametrize("splits", [1, 4])
@pytest.mark.parametrize("layout", LAYOUTS, ids=[f"tn{a}_ws{b}_pg{c}" for a, b, c in LAYOUTS])
def test_transposed_linear_layouts_match_oracle(layout, splits, knob):
    tn, ws, pg = layout
    knob("DS_JIT_TN", tn)
    knob("DS_JIT_WSPLIT", ws)
    knob("DS_JIT_PGROUPS", pg)
    n, c, k = 200, 700, 150
    codes, x, bias, _ = draw(zlib.crc32(repr((layout, splits)).encode()), n, c, k)
    say(f"jit linear layout {layout} splits={splits}")
    plan = ops.JitConv(ops.pack_shift_weights(codes), (n, c, 1, 1), 1, bias=bias, splits=splits)
    assert (plan.channels, plan.wsplit, plan.pixel_groups) == (tn, ws, pg)
    y = plan(to_dev(x.reshape(n, c, 1, 1))).cpu().numpy().reshape(n, k)
    plan.close()
    np.testing.assert_array_equal(y, oracle.linear_shift(x, codes, bias))


@pytest.mark.parametrize("act_bits", [16, 8])
def test_transposed_linear_narrow_activations(act_bits):
    n, c, k = 90, 333, 70
    codes, _, bias, rng = draw(act_bits, n, c, k)
    dt = {16: np.int16, 8: np.int8}[act_bits]
    info = np.iinfo(dt)
    x = rng.integers(info.min, info.max, (n, c), endpoint=True).astype(dt)
    say(f"jit linear act{act_bits}")
    plan = ops.JitConv(ops.pack_shift_weights(codes), (n, c, 1, 1), 1, bias=bias, act_bits=act_bits)
    y = plan(to_dev(x.reshape(n, c, 1, 1))).cpu().numpy().reshape(n, k)
    plan.close()
    np.testing.assert_array_equal(y, oracle.linear_shift(x.astype(np.int32), codes, bias))


def test_transposed_linear_multiplication_plan():
    n, c, k = 70, 200, 90
    rng = np.random.default_rng(77)
    w = rng.integers(-(2 ** 23), 2 ** 23, (k, c)).astype(np.int32)
    w[rng.random(w.shape) < 0.2] = 0
    x = rng.integers(-(2 ** 31), 2 ** 31, (n, c), dtype=np.int64).astype(np.int32)
    bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
    say("jit linear multiplication plan")
    plan = ops.JitConvMul(w, (n, c, 1, 1), 1, bias=bias)
    y = plan(to_dev(x.reshape(n, c, 1, 1))).cpu().numpy()
    plan.close()
    np.testing.assert_array_equal(y, oracle.conv2d_mul24(x.reshape(n, c, 1, 1), w, bias, r=1))


def test_transposed_linear_plan_runs_twice_on_new_inputs():
    n, c, k = 130, 64, 65
    codes, x, bias, rng = draw(5, n, c, k)
    plan = ops.JitConv(ops.pack_shift_weights(codes), (n, c, 1, 1), 1, bias=bias)
    for i in range(2):
        xi = x if i == 0 else rng.integers(-(2 ** 31), 2 ** 31, (n, c), dtype=np.int64).astype(np.int32)
        y = plan(to_dev(xi.reshape(n, c, 1, 1))).cpu().numpy().reshape(n, k)
        np.testing.assert_array_equal(y, oracle.linear_shift(xi, codes, bias))
    plan.close()


@pytest.mark.parametrize("splits", [0, 1, 3])
@pytest.mark.parametrize("shape", [(2, 7, 3), (33, 300, 70), (130, 97, 200), (256, 512, 300)],
                         ids=["2x7to3", "33x300to70", "130x97to200", "256x512to300"])
def test_transposed_linear_input_gradient_plans(shape, splits):
    """Input-gradient plans of a LinearShift (dx [n][c] = dy [n][k] through the
    codes): on dy^T, transposed back into dx."""
    n, c, k = shape
    rng = np.random.default_rng(zlib.crc32(repr((shape, splits)).encode()))
    codes = (rng.integers(0, 2, (k, c)) << 4 | rng.integers(0, 16, (k, c))).astype(np.uint8)
    dy = rng.integers(-(2 ** 31), 2 ** 31, (n, k), dtype=np.int64).astype(np.int32)
    say(f"jit linear input gradient {shape} splits={splits}")
    plan = ops.JitConvBackwardData(ops.pack_shift_weights(codes), (n, c, 1, 1), 1, splits=splits)
    dx = plan(to_dev(dy.reshape(n, k, 1, 1))).cpu().numpy().reshape(n, c)
    plan.close()
    np.testing.assert_array_equal(dx, oracle.linear_shift_backward_data(dy, codes))
