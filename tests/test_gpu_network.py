"""GPU parity of chained inference: the fused convolution epilogue, pooling, and a
whole ResNet-18 forward pass with shift convolutions, bit for bit against the oracle.

The fused epilogue runs in the convolution kernel's registers when a layer is not
split (and not transposed), and as a pass of its own otherwise; the cases below
cover both, the one-thread-per-output kernel, and the transposed 1 x 1 path.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops
from paper_1905_13298_amd import workloads as W
from paper_1905_13298_amd.network import ShiftNetwork
from paper_1905_13298_amd.workloads import random_codes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


# (n, c, h, k, r, stride, pad): fused in registers, split-K, transposed 1x1, strided 1x1, 7x7
FUSED_SHAPES = [(8, 16, 32, 64, 3, 1, 1), (3, 8, 40, 32, 1, 1, 0), (1, 256, 7, 64, 3, 1, 1),
                (4, 64, 1, 40, 1, 1, 0), (2, 32, 20, 48, 1, 2, 0), (4, 3, 30, 16, 7, 2, 3)]
COMBOS = ["relu", "affine", "affine_noadd", "residual", "all"]


@pytest.mark.parametrize("shape", FUSED_SHAPES)
@pytest.mark.parametrize("combo", COMBOS)
def test_fused_conv_matches_oracle(shape, combo):
    n, c, h, k, r, st, pd = shape
    say(f"fused conv {shape} {combo}: {ops.describe_conv2d(n, c, h, h, k, r, st, pd)}")
    rng = np.random.default_rng(zlib.crc32(repr((shape, combo)).encode()))
    x = rng.integers(-(2 ** 22), 2 ** 22, (n, c, h, h)).astype(np.int32)
    codes = random_codes(rng, (k, c * r * r), zero_frac=0.1)
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    oh = ops.out_size(h, pd, r, st)
    mul = add = res = None
    if combo in ("affine", "affine_noadd", "all"):
        mul = rng.integers(-(2 ** 18), 2 ** 18, k).astype(np.int32)
    if combo in ("affine", "all"):
        add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    if combo in ("residual", "all"):
        res = rng.integers(-(2 ** 24), 2 ** 24, (n, k, oh, oh)).astype(np.int32)
    relu = combo in ("relu", "all")
    wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    y = ops.conv2d_shift_fused(to_dev(x), wp, to_dev(bias), r, st, pd, mul=to_dev(mul),
                               add=to_dev(add), mul_shift=13, residual=to_dev(res), relu=relu)
    want = oracle.epilogue(oracle.conv2d_shift(x, codes, bias, r=r, stride=st, pad=pd), mul, add,
                           13, residual=res, relu=relu)
    np.testing.assert_array_equal(y.cpu().numpy(), want)


def test_fused_conv_direct_kernel(knob):
    knob("DS_FORCE_VARIANT", 0)
    n, c, h, k = 2, 5, 11, 7
    rng = np.random.default_rng(5)
    x = rng.integers(-(2 ** 22), 2 ** 22, (n, c, h, h)).astype(np.int32)
    codes = random_codes(rng, (k, c * 9))
    mul = rng.integers(1, 2 ** 17, k).astype(np.int32)
    add = rng.integers(-(2 ** 16), 2 ** 16, k).astype(np.int32)
    res = rng.integers(-(2 ** 20), 2 ** 20, (n, k, h, h)).astype(np.int32)
    assert ops.describe_conv2d(n, c, h, h, k, 3, 1, 1) == "direct"
    y = ops.conv2d_shift_fused(to_dev(x), to_dev(ops.pack_shift_weights(codes).view(np.int32)), None,
                               3, 1, 1, mul=to_dev(mul), add=to_dev(add), mul_shift=16,
                               residual=to_dev(res), relu=True)
    want = oracle.epilogue(oracle.conv2d_shift(x, codes, None, r=3, stride=1, pad=1), mul, add, 16,
                           residual=res, relu=True)
    np.testing.assert_array_equal(y.cpu().numpy(), want)


def test_relu_flag_on_plain_operators():
    rng = np.random.default_rng(6)
    x = rng.integers(-(2 ** 22), 2 ** 22, (16, 300)).astype(np.int32)
    codes = random_codes(rng, (70, 300))
    wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    y = ops.linear_shift(to_dev(x), wp, None, relu=True).cpu().numpy()
    np.testing.assert_array_equal(y, np.maximum(oracle.linear_shift(x, codes), 0))
    xc = rng.integers(-(2 ** 22), 2 ** 22, (2, 6, 13, 13)).astype(np.int32)
    cc = random_codes(rng, (9, 54))
    yc = ops.conv2d_shift(to_dev(xc), to_dev(ops.pack_shift_weights(cc).view(np.int32)), None, 3, 1, 1,
                          relu=True).cpu().numpy()
    np.testing.assert_array_equal(yc, np.maximum(oracle.conv2d_shift(xc, cc, None, r=3, stride=1, pad=1), 0))


@pytest.mark.parametrize("shape", [(4, 64, 112, 112, 3, 2, 1), (2, 5, 9, 7, 3, 2, 1), (1, 3, 8, 8, 2, 2, 0),
                                   (2, 4, 10, 10, 3, 1, 1), (1, 1, 1, 1, 1, 1, 0)])
def test_maxpool_matches_oracle(shape):
    n, c, h, w, r, st, pd = shape
    rng = np.random.default_rng(h * w + r)
    x = rng.integers(-(2 ** 31), 2 ** 31 - 1, (n, c, h, w), dtype=np.int64).astype(np.int32)
    y = ops.maxpool2d(to_dev(x), r, st, pd).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.maxpool2d(x, r=r, stride=st, pad=pd))


@pytest.mark.parametrize("shape", [(32, 512, 7, 7), (3, 5, 1, 1), (2, 7, 13, 11)])
def test_avgpool_matches_oracle(shape):
    rng = np.random.default_rng(sum(shape))
    x = rng.integers(-(2 ** 31), 2 ** 31 - 1, shape, dtype=np.int64).astype(np.int32)
    y = ops.avgpool2d_global(to_dev(x)).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.avgpool_global(x))


@pytest.mark.parametrize("jit", [False, "all"], ids=["runtime", "jit"])
def test_resnet18_forward_matches_oracle(jit):
    """Every intermediate buffer of a ResNet-18 forward pass (batch 2), bit for bit,
    with the runtime kernels and with weight-specialised plans."""
    n = 2
    graph, params = W.resnet18_graph(n), W.resnet18_params(n)
    x = W.gen_images(n)
    say(f"resnet18 forward n=2 jit={jit}")
    net = ShiftNetwork(graph, params, jit=jit)
    assert len(net.plans) == (21 if jit else 0)   # every conv (the 7 x 7 stem too) and the fc
    got = net.forward(to_dev(x), keep=True)
    want = oracle.network_forward(graph, params, x, keep=True)
    for op in graph:
        name = op["dst"]
        np.testing.assert_array_equal(got[name].cpu().numpy(), want[name], err_msg=name)
    # a second pass on the same buffers gives the same logits
    again = net.forward(to_dev(x)).cpu().numpy()
    np.testing.assert_array_equal(again, want["logits"])


def test_resnet18_forward_jit_full_batch_equals_runtime():
    """Batch 32 (the benchmark's): the logits and every block output of the plans'
    forward pass equal the runtime kernels' bit for bit."""
    n = 32
    graph, params = W.resnet18_graph(n), W.resnet18_params(n)
    x = to_dev(W.gen_images(n))
    say("resnet18 forward n=32 jit vs runtime")
    a = ShiftNetwork(graph, params).forward(x, keep=True)
    b = ShiftNetwork(graph, params, jit=True).forward(x, keep=True)
    for op in graph:
        assert torch.equal(a[op["dst"]], b[op["dst"]]), op["dst"]
