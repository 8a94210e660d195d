"""GPU parity: the HIP path against the oracle, bit for bit.

Every case runs the library through its C ABI (via ``paper_1905_13298_amd.ops``)
on seeded inputs and compares the int32 outputs with the oracle element by
element. Small batches of the benchmark layers are checked here; every layer at the
benchmark batch is checked in full in test_gpu_full_oracle.
"""
import re
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import _native, ops
from paper_1905_13298_amd import workloads as W
from paper_1905_13298_amd.workloads import random_codes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
I32_MIN, I32_MAX = -(2 ** 31), 2 ** 31 - 1


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def gpu_layer(layer, x, codes, bias, out=None):
    wp = ops.pack_shift_weights(codes).view(np.int32)
    xt, wt, bt = to_dev(x), to_dev(wp), to_dev(bias)
    if layer.kind == "linear":
        y = ops.linear_shift(xt, wt, bt, out=out)
    else:
        y = ops.conv2d_shift(xt, wt, bt, (layer.r, layer.s), layer.stride, layer.pad, out=out)
    return y


def oracle_layer(layer, x, codes, bias):
    if layer.kind == "linear":
        return oracle.linear_shift(x, codes, bias)
    return oracle.conv2d_shift(x, codes, bias, r=layer.r, s=layer.s, stride=layer.stride,
                               pad=layer.pad)


def oracle_points(layer, x, codes, bias, idx):
    if layer.kind == "linear":
        return oracle.linear_shift_points(x, codes, bias, idx)
    return oracle.conv2d_shift_points(x, codes, bias, idx, r=layer.r, s=layer.s,
                                      stride=layer.stride, pad=layer.pad)


def sample_indices(layer, rng, count):
    """Random outputs plus the first/last element of every pixel tile boundary region."""
    total = int(np.prod(layer.y_shape))
    idx = set(rng.choice(total, size=min(count, total), replace=False).tolist())
    idx.update([0, total - 1])
    ohow = layer.oh * layer.ow
    for k in (0, layer.k - 1):
        for q in (0, 63, 64, 255, 256, 511, 512, layer.n * ohow - 1):
            if q < layer.n * ohow:
                n, p = divmod(q, ohow)
                idx.add((n * layer.k + k) * ohow + p)
    return np.array(sorted(idx), dtype=np.int64)


def check_full(layer, x, codes, bias, what):
    y = gpu_layer(layer, x, codes, bias).cpu().numpy()
    want = oracle_layer(layer, x, codes, bias)
    bad = np.flatnonzero(y.ravel() != want.ravel())
    assert bad.size == 0, f"{what}: {bad.size} mismatches, first at {bad[:5]}"


# ---------------------------------------------------------------------------
# the five workloads


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_single_layer_configs_exact(cfg):
    (layer,) = W.config_layers(cfg)
    x, codes, bias = W.gen_layer(layer, W.CONFIG_SEEDS[cfg], 0)
    say(f"{W.CONFIG_NAMES[cfg]} {layer}")
    check_full(layer, x, codes, bias, W.CONFIG_NAMES[cfg])


@pytest.mark.parametrize("cfg,batch", [(3, 2), (4, 2)])
def test_network_layers_small_batch_exact(cfg, batch):
    for li, layer in enumerate(W.config_layers(cfg)):
        small = layer.with_batch(batch)
        x, codes, bias = W.gen_layer(small, W.CONFIG_SEEDS[cfg], li)
        say(f"{W.CONFIG_NAMES[cfg]} layer {li} {small.name} n={batch}")
        check_full(small, x, codes, bias, f"{W.CONFIG_NAMES[cfg]}/{small.name}")


# ---------------------------------------------------------------------------
# edge shapes


EDGE = [
    # name, N, C, H, W, K, r, s, stride, pad
    ("ragged_k_c_pix", 3, 13, 9, 11, 37, 3, 3, 1, 1),
    ("c3_stem_like", 2, 3, 23, 23, 10, 7, 7, 2, 3),
    ("1x1_s2", 3, 20, 15, 15, 33, 1, 1, 2, 0),
    ("1x1_s1_odd", 2, 9, 7, 5, 70, 1, 1, 1, 0),
    ("1x1_pad", 1, 5, 6, 6, 9, 1, 1, 1, 1),
    ("3x3_s2_odd", 2, 11, 13, 9, 17, 3, 3, 2, 1),
    ("3x3_s3_pad2", 1, 6, 17, 17, 8, 3, 3, 3, 2),
    ("rect_2x3", 2, 5, 10, 12, 6, (2, 3), None, (1, 2), (0, 1)),
    ("5x5", 1, 4, 12, 12, 9, 5, 5, 1, 2),
    ("4x4", 1, 3, 9, 9, 5, 4, 4, 1, 1),
    ("6x6_direct", 1, 3, 12, 12, 5, 6, 6, 1, 1),
    ("7x7_images", 5, 16, 7, 7, 40, 3, 3, 1, 1),
    ("batch1_1x1_image", 1, 64, 1, 1, 10, 1, 1, 1, 0),
    ("tiny", 1, 1, 1, 1, 1, 1, 1, 1, 0),
    ("big_c_small_k", 1, 300, 6, 6, 3, 3, 3, 1, 1),
]


def edge_case(spec, signed, seed):
    name, N, C, H, Wd, K, r, s, stride, pad = spec
    if isinstance(r, tuple):
        r, s = r
    s = r if s is None else s
    rng = np.random.default_rng(seed)
    lo = -(2 ** 24) if signed else 0
    x = rng.integers(lo, 2 ** 24, (N, C, H, Wd)).astype(np.int32)
    codes = random_codes(rng, (K, C * r * s), zero_frac=0.2)
    bias = rng.integers(-(2 ** 20), 2 ** 20, K).astype(np.int32) if seed % 2 else None
    return x, codes, bias, r, s, stride, pad


@pytest.mark.parametrize("signed", [False, True])
@pytest.mark.parametrize("spec", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes_exact(spec, signed):
    x, codes, bias, r, s, stride, pad = edge_case(spec, signed, zlib.crc32(spec[0].encode()) % 1000 + signed)
    xt, bt = to_dev(x), to_dev(bias)
    wt = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    y = ops.conv2d_shift(xt, wt, bt, (r, s), stride, pad).cpu().numpy()
    want = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=stride, pad=pad)
    np.testing.assert_array_equal(y, want)


@pytest.mark.parametrize("shape", [(1, 1, 1), (1, 7, 5), (3, 100, 33), (300, 70, 65),
                                   (257, 129, 31), (16, 4096, 8)])
@pytest.mark.parametrize("signed", [False, True])
def test_linear_shapes_exact(shape, signed):
    B, I, O = shape
    rng = np.random.default_rng(B * 7 + I + O + signed)
    lo = -(2 ** 20) if signed else 0
    x = rng.integers(lo, 2 ** 20, (B, I)).astype(np.int32)
    codes = random_codes(rng, (O, I), zero_frac=0.15)
    bias = rng.integers(-(2 ** 16), 2 ** 16, O).astype(np.int32)
    y = ops.linear_shift(to_dev(x), to_dev(ops.pack_shift_weights(codes).view(np.int32)),
                         to_dev(bias)).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.linear_shift(x, codes, bias))


def test_int32_extremes_wrap():
    rng = np.random.default_rng(5)
    x = rng.integers(I32_MIN, I32_MAX, (2, 8, 10, 10), endpoint=True).astype(np.int32)
    x[0, 0, 0, :4] = [I32_MIN, I32_MAX, -1, 0]
    codes = rng.integers(0, 32, (20, 72)).astype(np.uint8)
    codes[0, :] = 0  # +2^0 everywhere: sums wrap
    bias = rng.integers(I32_MIN, I32_MAX, 20, endpoint=True).astype(np.int32)
    y = ops.conv2d_shift(to_dev(x), to_dev(ops.pack_shift_weights(codes).view(np.int32)),
                         to_dev(bias), 3, 1, 1).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.conv2d_shift(x, codes, bias, r=3, pad=1))


def test_mixed_sign_chunks():
    """Negative inputs only in some input channels: chunks take different paths."""
    rng = np.random.default_rng(9)
    x = rng.integers(0, 2 ** 22, (2, 40, 12, 12)).astype(np.int32)
    x[:, 17] = -x[:, 17]
    x[1, 33, 5, 5] = -1
    codes = random_codes(rng, (24, 40 * 9), zero_frac=0.3)
    y = ops.conv2d_shift(to_dev(x), to_dev(ops.pack_shift_weights(codes).view(np.int32)),
                         None, 3, 1, 1).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.conv2d_shift(x, codes, None, r=3, pad=1))
    xl = rng.integers(0, 2 ** 22, (64, 100)).astype(np.int32)
    xl[3, 50] = -5
    cl = random_codes(rng, (50, 100), zero_frac=0.3)
    yl = ops.linear_shift(to_dev(xl), to_dev(ops.pack_shift_weights(cl).view(np.int32))).cpu().numpy()
    np.testing.assert_array_equal(yl, oracle.linear_shift(xl, cl, None))


# ---------------------------------------------------------------------------
# semantics band, buffers, streams


def test_output_canaries_untouched():
    rng = np.random.default_rng(3)
    for (n, c, h, w, k, r, st, pd) in [(2, 9, 11, 13, 21, 3, 1, 1), (3, 16, 8, 8, 40, 1, 2, 0)]:
        x = rng.integers(0, 2 ** 20, (n, c, h, w)).astype(np.int32)
        codes = random_codes(rng, (k, c * r * r))
        oh = (h + 2 * pd - r) // st + 1
        ow = (w + 2 * pd - r) // st + 1
        size = n * k * oh * ow
        big = torch.full((size + 2048,), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
        out = big[1024:1024 + size].view(n, k, oh, ow)
        ops.conv2d_shift(to_dev(x), to_dev(ops.pack_shift_weights(codes).view(np.int32)), None,
                         r, st, pd, out=out)
        b = big.cpu().numpy()
        assert np.all(b[:1024] == 0x5A5A5A5A) and np.all(b[1024 + size:] == 0x5A5A5A5A)
        np.testing.assert_array_equal(out.cpu().numpy(),
                                      oracle.conv2d_shift(x, codes, None, r=r, stride=st, pad=pd))


@pytest.mark.parametrize("offset", [0, 1], ids=["aligned", "offset_4_bytes"])
def test_split_outputs_ragged_and_unaligned(offset):
    """Split reductions whose output count is not a multiple of 4, written into a
    buffer on a 16-byte boundary and 4 bytes past one: the fill pass before the
    atomics in its vector form with its tail, and in its element-wise form; the
    runtime kernel and a plan with a forced split, both against the oracle, with
    canaries on both sides of y."""
    rng = np.random.default_rng(77 + offset)
    n, c, h, w, k = 1, 256, 7, 7, 255
    assert int(re.search(r"splits(\d+)", ops.describe_conv2d(n, c, h, w, k, 3, 1, 1)).group(1)) > 1
    x = rng.integers(0, 2 ** 20, (n, c, h, w)).astype(np.int32)
    codes = random_codes(rng, (k, c * 9), zero_frac=0.2)
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    want = oracle.conv2d_shift(x, codes, bias, r=3, s=3, stride=1, pad=1)
    size = want.size
    assert size % 4 == 3
    wp = ops.pack_shift_weights(codes)
    xt, bt = to_dev(x), to_dev(bias)
    plan = ops.JitConv(wp, x.shape, 3, 1, 1, bias=bias, splits=2)
    try:
        assert plan.splits == 2
        for name, run in [("runtime", lambda out: ops.conv2d_shift(xt, to_dev(wp.view(np.int32)), bt, 3,
                                                                   1, 1, out=out)),
                          ("plan", lambda out: plan(xt, out=out))]:
            big = torch.full((size + 2048,), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
            lo = 1024 + offset
            out = big[lo:lo + size].view(want.shape)
            run(out)
            b = big.cpu().numpy()
            say(name, "offset", offset)
            assert np.all(b[:lo] == 0x5A5A5A5A) and np.all(b[lo + size:] == 0x5A5A5A5A), name
            np.testing.assert_array_equal(b[lo:lo + size].reshape(want.shape), want, err_msg=name)
    finally:
        plan.close()


def test_padded_copy_ragged():
    """A plan reading a 5 x 5 window through its zero-padded copy of x, whose
    element count (3 planes of 13 x 13) is not a multiple of 4: the copy's vector
    stores and its tail, against the oracle."""
    rng = np.random.default_rng(5)
    x = rng.integers(-(2 ** 20), 2 ** 20, (1, 3, 9, 9)).astype(np.int32)
    codes = random_codes(rng, (7, 3 * 25), zero_frac=0.2)
    want = oracle.conv2d_shift(x, codes, None, r=5, s=5, stride=1, pad=2)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, 5, 1, 2)
    try:
        np.testing.assert_array_equal(plan(to_dev(x)).cpu().numpy(), want)
    finally:
        plan.close()


def test_nondefault_stream_and_repeat():
    rng = np.random.default_rng(4)
    x = rng.integers(0, 2 ** 20, (4, 32, 14, 14)).astype(np.int32)
    codes = random_codes(rng, (64, 32 * 9))
    want = oracle.conv2d_shift(x, codes, None, r=3, pad=1)
    xt = to_dev(x)
    wt = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    s = torch.cuda.Stream(DEV)
    with torch.cuda.stream(s):
        ys = [ops.conv2d_shift(xt, wt, None, 3, 1, 1) for _ in range(3)]
    s.synchronize()
    for y in ys:
        np.testing.assert_array_equal(y.cpu().numpy(), want)


def test_device_buffer_errors_write_nothing():
    lib = _native.lib()
    x = torch.zeros((2, 8), dtype=torch.int32, device=DEV)
    w = to_dev(ops.pack_shift_weights(np.zeros((4, 8), np.uint8)).view(np.int32))
    y = torch.full((2, 4), 7, dtype=torch.int32, device=DEV)
    # declared batch larger than the buffers
    st = lib.ds_linear_shift(x.data_ptr(), w.data_ptr(), None, y.data_ptr(), 1 << 24, 8, 4, 16, 0,
                             None)
    assert st == 3
    # host pointer for x
    xh = np.zeros((2, 8), np.int32)
    st = lib.ds_linear_shift(xh.ctypes.data, w.data_ptr(), None, y.data_ptr(), 2, 8, 4, 16, 0, None)
    assert st == 3
    torch.cuda.synchronize()
    assert torch.all(y == 7)


# ---------------------------------------------------------------------------
# the multiplication-based comparison kernels


@pytest.mark.parametrize("shape", [(2, 9, 11, 13, 21, 3, 1, 1), (3, 16, 8, 8, 40, 1, 2, 0),
                                   (1, 3, 30, 30, 8, 7, 2, 3), (2, 64, 14, 14, 64, 3, 1, 1)])
def test_mul_comparison_exact(shape):
    n, c, h, w, k, r, st, pd = shape
    rng = np.random.default_rng(sum(shape))
    x = rng.integers(-(2 ** 20), 2 ** 20, (n, c, h, w)).astype(np.int32)
    wt = rng.integers(-(2 ** 12), 2 ** 12, (k, c * r * r)).astype(np.int32)
    b = rng.integers(-99, 99, k).astype(np.int32)
    y = ops.conv2d_mul_i32(to_dev(x), to_dev(wt), to_dev(b), r, st, pd).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.conv2d_mul(x, wt, b, r=r, stride=st, pad=pd))
    xl = rng.integers(-(2 ** 20), 2 ** 20, (33, 70)).astype(np.int32)
    wl = rng.integers(I32_MIN, I32_MAX, (45, 70), endpoint=True).astype(np.int32)
    yl = ops.linear_mul_i32(to_dev(xl), to_dev(wl)).cpu().numpy()
    want = oracle.conv2d_mul(xl.reshape(33, 70, 1, 1), wl, None, r=1).reshape(33, 45)
    np.testing.assert_array_equal(yl, want)


@pytest.mark.parametrize("shape", [(2, 9, 11, 13, 21, 3, 1, 1), (3, 16, 8, 8, 40, 1, 2, 0),
                                   (1, 3, 30, 30, 8, 7, 2, 3), (2, 64, 14, 14, 64, 3, 1, 1)])
def test_mul24_comparison_exact(shape):
    """DS_MUL_I24: each product of the low 24 bits of x and w as signed values,
    on inputs that exceed 24 bits (the upper bits must be ignored) and on the
    LinearShift shape."""
    n, c, h, w, k, r, st, pd = shape
    rng = np.random.default_rng(sum(shape) + 24)
    x = rng.integers(I32_MIN, I32_MAX, (n, c, h, w), endpoint=True).astype(np.int32)
    wt = rng.integers(I32_MIN, I32_MAX, (k, c * r * r), endpoint=True).astype(np.int32)
    b = rng.integers(-99, 99, k).astype(np.int32)
    y = ops.conv2d_mul_i32(to_dev(x), to_dev(wt), to_dev(b), r, st, pd, mul24=True).cpu().numpy()
    np.testing.assert_array_equal(y, oracle.conv2d_mul24(x, wt, b, r=r, stride=st, pad=pd))
    xl = rng.integers(I32_MIN, I32_MAX, (33, 70), endpoint=True).astype(np.int32)
    wl = rng.integers(I32_MIN, I32_MAX, (45, 70), endpoint=True).astype(np.int32)
    yl = ops.linear_mul_i32(to_dev(xl), to_dev(wl), mul24=True).cpu().numpy()
    want = oracle.conv2d_mul24(xl.reshape(33, 70, 1, 1), wl, None, r=1).reshape(33, 45)
    np.testing.assert_array_equal(yl, want)
