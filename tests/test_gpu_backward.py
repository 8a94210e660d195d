"""GPU parity of the input gradients (``ds_conv2d_shift_backward_data``,
``ds_linear_shift_backward_data``) with the oracle, bit for bit.

Edge shapes cover every path of the stride-phase decomposition: stride 1 (one
phase), strides 2 and 3 with padding (phases with 1 and 2 taps per axis,
pointwise and window staging, split and unsplit), phases no tap reaches (zero
fill), rectangular windows and strides, and shapes that go to the gather
kernel (a phase with padding beyond its window; a window width without a
tiled instance); the gather kernel is also forced on its own. Gradients are
signed int32 over the whole range. At full size, the input gradient of every
ResNet-50 convolution (batch 128) equals the gather kernel element by element,
and 400 sampled elements per layer equal the oracle's.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops
from paper_1905_13298_amd import workloads as W
from paper_1905_13298_amd.workloads import random_codes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def oh_of(h, pad, r, stride):
    return (h + 2 * pad - r) // stride + 1


def pair(v):
    return (v, v) if np.isscalar(v) else tuple(v)


# name, n, c, h, w, k, r, s, stride, pad
EDGE = [
    ("s1_3x3", 2, 13, 9, 11, 37, 3, 3, 1, 1),
    ("s1_3x3_pad0", 2, 6, 8, 8, 9, 3, 3, 1, 0),
    ("s1_3x3_pad2", 1, 5, 7, 7, 6, 3, 3, 1, 2),
    ("s2_3x3_even", 3, 20, 16, 16, 33, 3, 3, 2, 1),
    ("s2_3x3_odd", 2, 11, 13, 9, 17, 3, 3, 2, 1),
    ("s2_3x3_pad0", 2, 7, 11, 11, 10, 3, 3, 2, 0),
    ("s3_3x3_pad1", 1, 6, 17, 17, 8, 3, 3, 3, 1),
    ("s2_1x1", 3, 20, 15, 15, 33, 1, 1, 2, 0),
    ("s2_1x1_even", 2, 64, 14, 14, 70, 1, 1, 2, 0),
    ("s1_1x1", 2, 9, 7, 5, 70, 1, 1, 1, 0),
    ("rect_2x3", 2, 5, 10, 12, 6, (2, 3), (2, 3), 1, 1),
    ("rect_stride", 2, 5, 9, 8, 3, (2, 3), (2, 3), (2, 1), (1, 0)),   # negative-pad phase: gather
    ("s2_7x7_stem", 2, 3, 30, 30, 16, 7, 7, 2, 3),                    # 3- and 4-tap phases; plans: padded
    ("pad_beyond_1x1", 1, 3, 6, 6, 2, 1, 1, 1, 1),                    # gather
    ("big_k_small_c", 2, 3, 12, 12, 300, 3, 3, 2, 1),
    ("many_tiles", 4, 64, 20, 20, 128, 3, 3, 1, 1),
    ("tiny", 1, 1, 1, 1, 1, 1, 1, 1, 0),
]


def make(seed, n, c, h, w, k, r, s, st, pd, lim=2 ** 31):
    r, s = pair(r) if not np.isscalar(r) else (r, s)
    sh, sw = pair(st)
    ph, pw = pair(pd)
    rng = np.random.default_rng(seed)
    oh, ow = oh_of(h, ph, r, sh), oh_of(w, pw, s, sw)
    dy = rng.integers(-lim, lim, (n, k, oh, ow), dtype=np.int64).astype(np.int32)
    codes = rng.integers(0, 32, (k, c * r * s)).astype(np.uint8)
    return dy, codes, (r, s)


@pytest.mark.parametrize("direct", [False, True], ids=["auto", "gather"])
@pytest.mark.parametrize("spec", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes_match_oracle(spec, direct, knob):
    name, n, c, h, w, k, r, s, st, pd = spec
    if direct:
        knob("DS_FORCE_VARIANT", 0)
    rr = r if np.isscalar(r) else r[0]
    ss = s if np.isscalar(s) else s[1]
    dy, codes, _ = make(zlib.crc32(name.encode()), n, c, h, w, k, rr, ss, st, pd)
    plan = ops.describe_conv2d_backward_data(n, c, h, w, k, (rr, ss), st, pd)
    say(f"backward {name} direct={direct}: {plan}")
    wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    dx = ops.conv2d_shift_backward_data(to_dev(dy), wp, (n, c, h, w), (rr, ss), st, pd).cpu().numpy()
    want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, w), r=rr, s=ss, stride=st, pad=pd)
    bad = np.flatnonzero(dx.ravel() != want.ravel())
    assert bad.size == 0, f"{bad.size} of {want.size} differ, first at {bad[:5]}"


def test_plans_cover_the_expected_paths():
    d = ops.describe_conv2d_backward_data
    assert d(2, 64, 56, 56, 128, 3, 2, 1).startswith("phases4")
    assert d(2, 64, 56, 56, 64, 3, 1, 1).startswith("phases1")
    assert "zero" in d(8, 64, 14, 14, 70, 1, 2, 0)
    assert d(2, 5, 9, 8, 3, (2, 3), (2, 1), (1, 0)) == "direct"
    stem = d(2, 3, 30, 30, 16, 7, 2, 3)
    assert stem.startswith("phases4") and stem.count("tiled") == 4


@pytest.mark.parametrize("shape", [(8, 256, 128), (33, 300, 70), (256, 4096, 4096), (1, 1, 1)])
def test_linear_matches_oracle(shape):
    batch, fin, fout = shape
    rng = np.random.default_rng(fin + fout)
    dy = rng.integers(-(2 ** 31), 2 ** 31, (batch, fout), dtype=np.int64).astype(np.int32)
    codes = random_codes(rng, (fout, fin), zero_frac=0.1)
    wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    say(f"linear backward {shape}")
    dx = ops.linear_shift_backward_data(to_dev(dy), wp, fin).cpu().numpy()
    np.testing.assert_array_equal(dx, oracle.linear_shift_backward_data(dy, codes))


def test_output_fully_overwritten_and_repeatable():
    """dx starts as garbage; every element is written, and a second call gives the same."""
    n, c, h, w, k = 2, 16, 14, 14, 24
    dy, codes, _ = make(77, n, c, h, w, k, 3, 3, 2, 1)
    wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, w), r=3, stride=2, pad=1)
    out = torch.full((n, c, h, w), -123456, dtype=torch.int32, device=DEV)
    for _ in range(2):
        ops.conv2d_shift_backward_data(to_dev(dy), wp, (n, c, h, w), 3, 2, 1, out=out)
        np.testing.assert_array_equal(out.cpu().numpy(), want)


@pytest.mark.parametrize("offset", [0, 1, 2, 3])
def test_cleared_positions_at_any_alignment(offset):
    """A 1x1 stride-2 layer: dx is cleared densely (16-byte stores on the aligned
    part, single stores around it) before the phase writes its positions; dx views
    at every 4-byte offset, with guard elements around them left untouched, on
    both paths."""
    n, c, h, w, k = 3, 20, 15, 13, 33
    dy, codes, _ = make(91 + offset, n, c, h, w, k, 1, 1, 2, 0)
    wph = ops.pack_shift_weights(codes)
    wp = to_dev(wph.view(np.int32))
    want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, w), r=1, stride=2, pad=0)
    size = n * c * h * w
    plan = ops.JitConvBackwardData(wph, (n, c, h, w), 1, 2, 0)
    for run in ("runtime", "plan"):
        big = torch.full((size + 8,), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
        out = big[offset:offset + size].view(n, c, h, w)
        if run == "runtime":
            ops.conv2d_shift_backward_data(to_dev(dy), wp, (n, c, h, w), 1, 2, 0, out=out)
        else:
            plan(to_dev(dy), out=out)
        got = big.cpu().numpy()
        np.testing.assert_array_equal(got[offset:offset + size].reshape(want.shape), want, err_msg=run)
        assert np.all(got[:offset] == 0x5A5A5A5A) and np.all(got[offset + size:] == 0x5A5A5A5A), run
    plan.close()


def test_errors_write_nothing():
    n, c, h, w, k = 1, 4, 6, 6, 5
    dy = torch.zeros((n, k, 6, 6), dtype=torch.int32, device=DEV)
    wp = to_dev(ops.pack_shift_weights(np.zeros((k, c * 9), np.uint8)).view(np.int32))
    dx = torch.full((n, c, h, w), 7, dtype=torch.int32, device=DEV)
    with pytest.raises(ops.DeepShiftError, match="INVALID_ARG"):
        ops.call("ds_conv2d_shift_backward_data", dy.data_ptr(), wp.data_ptr(), dx.data_ptr(),
                 n, c, h, w, k, 3, 3, 1, 1, 1, 1, 16, 1, None)                     # flags
    with pytest.raises(ops.DeepShiftError, match="INVALID_ARG"):
        ops.conv2d_shift_backward_data(dy, wp, (n, c, h, w), 3, 1, 1,
                                       out=dy.view(-1)[: n * c * h * w].view(n, c, h, w))  # overlap
    with pytest.raises(ops.DeepShiftError, match="INVALID_SHAPE"):
        ops.conv2d_shift_backward_data(dy, wp, (n, c, 2, 2), 3, 1, 0, out=dx[:, :, :2, :2].contiguous())
    assert torch.all(dx == 7)


def test_resnet50_full_batch_against_gather_kernel_and_oracle(knob):
    """Every ResNet-50 convolution at batch 128 (the stem aside: an input gradient of
    the images is not needed): all elements equal the gather kernel's, 400 sampled
    elements per layer equal the oracle's."""
    rng = np.random.default_rng(51)
    layers = W.config_layers(4)
    for li, L in enumerate(layers):
        if L.kind != "conv" or L.name == "conv1":
            continue
        codes = W.gen_codes(L, W.CONFIG_SEEDS[4], li)
        g = np.random.default_rng([4, li, 7])
        dy = np.rint(g.standard_normal(L.y_shape, dtype=np.float32) * 2 ** 16).astype(np.int32)
        wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
        dyd = to_dev(dy)
        x_shape = L.x_shape
        say(f"backward resnet50 {L.name}: {ops.describe_conv2d_backward_data(*x_shape, L.k, (L.r, L.s), L.stride, L.pad)}")
        dx = ops.conv2d_shift_backward_data(dyd, wp, x_shape, (L.r, L.s), L.stride, L.pad)
        knob("DS_FORCE_VARIANT", 0)
        ref = ops.conv2d_shift_backward_data(dyd, wp, x_shape, (L.r, L.s), L.stride, L.pad)
        knob("DS_FORCE_VARIANT", -1)
        diff = int((dx != ref).sum())
        assert diff == 0, f"{L.name}: {diff} elements differ from the gather kernel"
        total = int(np.prod(x_shape))
        idx = np.unique(np.concatenate([rng.choice(total, 400, replace=False), [0, total - 1]]))
        got = dx.reshape(-1)[torch.from_numpy(idx).to(DEV)].cpu().numpy()
        want = oracle.conv2d_shift_backward_data_points(dy, codes, x_shape, idx, r=L.r, s=L.s,
                                                        stride=L.stride, pad=L.pad)
        np.testing.assert_array_equal(got, want, err_msg=L.name)
        del dx, ref, dyd


def test_stem_gradient_on_tiled_phases_full_size(knob):
    """The 7 x 7 / 2 stem's input gradient at 224 x 224 (batch 4) on the runtime
    path: four stride phases of 3 and 4 taps per row on the tiled kernel. All
    elements equal the gather kernel's and the plan's, 400 sampled elements the
    oracle's."""
    L = W.config_layers(4)[0]
    n = 4
    x_shape = (n,) + tuple(L.x_shape[1:])
    codes = W.gen_codes(L, W.CONFIG_SEEDS[4], 0)
    g = np.random.default_rng(17)
    dy = np.rint(g.standard_normal((n, L.k) + tuple(L.y_shape[2:]), dtype=np.float32) * 2 ** 16).astype(np.int32)
    path = ops.describe_conv2d_backward_data(*x_shape, L.k, (L.r, L.s), L.stride, L.pad)
    assert path.startswith("phases4") and path.count("tiled") == 4, path
    say(f"backward stem {x_shape}: {path}")
    wp = to_dev(ops.pack_shift_weights(codes).view(np.int32))
    dyd = to_dev(dy)
    dx = ops.conv2d_shift_backward_data(dyd, wp, x_shape, (L.r, L.s), L.stride, L.pad)
    knob("DS_FORCE_VARIANT", 0)
    ref = ops.conv2d_shift_backward_data(dyd, wp, x_shape, (L.r, L.s), L.stride, L.pad)
    knob("DS_FORCE_VARIANT", -1)
    assert int((dx != ref).sum()) == 0
    plan = ops.JitConvBackwardData(ops.pack_shift_weights(codes), x_shape, (L.r, L.s), L.stride, L.pad)
    assert int((plan(dyd) != dx).sum()) == 0
    plan.close()
    total = int(np.prod(x_shape))
    idx = np.unique(np.concatenate([np.random.default_rng(3).choice(total, 400, replace=False), [0, total - 1]]))
    got = dx.reshape(-1)[torch.from_numpy(idx).to(DEV)].cpu().numpy()
    want = oracle.conv2d_shift_backward_data_points(dy, codes, x_shape, idx, r=L.r, s=L.s, stride=L.stride,
                                                    pad=L.pad)
    np.testing.assert_array_equal(got, want)


JIT_EDGE = EDGE


@pytest.mark.parametrize("splits", [0, 1, 3])
@pytest.mark.parametrize("spec", JIT_EDGE, ids=[e[0] for e in JIT_EDGE])
def test_weight_specialised_plans_match_oracle(spec, splits):
    """Input-gradient plans (one generated kernel per stride phase, writing its rows
    and columns of dx through an output map) against the oracle."""
    name, n, c, h, w, k, r, s, st, pd = spec
    rr = r if np.isscalar(r) else r[0]
    ss = s if np.isscalar(s) else s[1]
    dy, codes, _ = make(zlib.crc32(name.encode()) + 7, n, c, h, w, k, rr, ss, st, pd)
    plan = ops.JitConvBackwardData(ops.pack_shift_weights(codes), (n, c, h, w), (rr, ss), st, pd,
                                   splits=splits)
    say(f"jit backward {name} splits={splits}: {plan.segments} segments, {plan.code_bytes} code bytes")
    out = torch.full((n, c, h, w), 0x5A5A5A5A, dtype=torch.int32, device=DEV)   # every element written
    dx = plan(to_dev(dy), out=out).cpu().numpy()
    want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, w), r=rr, s=ss, stride=st, pad=pd)
    bad = np.flatnonzero(dx.ravel() != want.ravel())
    assert bad.size == 0, f"{bad.size} of {want.size} differ, first at {bad[:5]}"
    plan.close()


def test_stride_phases_fuse_into_one_kernel():
    """A 3x3 stride-2 layer's four phases become one kernel of 4 x ceil(c/64) output-
    channel groups (no split); with odd extents (phase grids differ) or a forced split
    each phase keeps a kernel of its own. Each plan is checked against the oracle."""
    for (h, splits, segments) in ((16, 0, 4 * 2), (16, 3, 4 * 2 * 3), (15, 0, None)):
        n, c, k = 2, 70, 33
        dy, codes, _ = make(1234 + h + splits, n, c, h, h, k, 3, 3, 2, 1)
        plan = ops.JitConvBackwardData(ops.pack_shift_weights(codes), (n, c, h, h), 3, 2, 1,
                                       splits=splits)
        say(f"fuse h={h} splits={splits}: {plan.segments} segments, {plan.splits} parts")
        if segments is not None:
            assert plan.segments == segments
        dx = plan(to_dev(dy)).cpu().numpy()
        plan.close()
        want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, h), r=3, stride=2, pad=1)
        np.testing.assert_array_equal(dx, want)


def test_weight_specialised_plan_limits_and_arguments():
    codes = np.zeros((16, 1024), np.uint8)      # a phase window 1024 columns wide
    with pytest.raises(ops.DeepShiftError, match="UNSUPPORTED"):
        ops.JitConvBackwardData(ops.pack_shift_weights(codes), (2, 1, 4, 1030), (1, 1024), 1, 0)
    codes = random_codes(np.random.default_rng(3), (8, 4 * 9))
    plan = ops.JitConvBackwardData(ops.pack_shift_weights(codes), (2, 4, 8, 8), 3, 2, 1)
    dy = torch.zeros(plan.x_shape, dtype=torch.int32, device=DEV)
    with pytest.raises(ops.DeepShiftError, match="residual must be NULL"):
        plan(dy, residual=torch.zeros(plan.y_shape, dtype=torch.int32, device=DEV))
    with pytest.raises(ops.DeepShiftError, match="overlaps"):
        big = torch.zeros(4 * 8 * 8 * 2 + 64, dtype=torch.int32, device=DEV)
        plan(big[: dy.numel()].view(plan.x_shape), out=big[:2 * 4 * 8 * 8].view(plan.y_shape))
    plan.close()


def test_linear_plan_matches_oracle():
    rng = np.random.default_rng(61)
    dy = rng.integers(-(2 ** 31), 2 ** 31, (33, 70), dtype=np.int64).astype(np.int32)
    codes = random_codes(rng, (70, 300))
    plan = ops.JitConvBackwardData(ops.pack_shift_weights(codes), (33, 300, 1, 1), 1)
    dx = plan(to_dev(dy.reshape(33, 70, 1, 1))).cpu().numpy().reshape(33, 300)
    np.testing.assert_array_equal(dx, oracle.linear_shift_backward_data(dy, codes))
    plan.close()


def test_resnet50_full_batch_plans_equal_runtime_kernel():
    """Every ResNet-50 convolution but the stem at batch 128: the plans' input
    gradient equals ds_conv2d_shift_backward_data's on every element."""
    layers = W.config_layers(4)
    for li, L in enumerate(layers):
        if L.kind != "conv" or L.name == "conv1":
            continue
        codes = W.gen_codes(L, W.CONFIG_SEEDS[4], li)
        g = np.random.default_rng([4, li, 7])
        dy = to_dev(np.rint(g.standard_normal(L.y_shape, dtype=np.float32) * 2 ** 16).astype(np.int32))
        wp = ops.pack_shift_weights(codes)
        plan = ops.JitConvBackwardData(wp, L.x_shape, (L.r, L.s), L.stride, L.pad)
        say(f"jit backward resnet50 {L.name}: {plan.segments} segments, {plan.code_bytes / 2 ** 20:.1f} MiB")
        got = plan(dy)
        ref = ops.conv2d_shift_backward_data(dy, to_dev(wp.view(np.int32)), L.x_shape, (L.r, L.s),
                                             L.stride, L.pad)
        diff = int((got != ref).sum())
        assert diff == 0, f"{L.name}: {diff} elements differ"
        plan.close()
        del got, ref, dy


def _random_layers(count, seed):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        n, c, k = int(rng.integers(1, 4)), int(rng.integers(1, 150)), int(rng.integers(1, 150))
        r, s = int(rng.integers(1, 8)), int(rng.integers(1, 8))
        st, pd = int(rng.integers(1, 4)), int(rng.integers(0, 4))
        h, w = int(rng.integers(1, 26)), int(rng.integers(1, 26))
        if h + 2 * pd < r or w + 2 * pd < s:
            continue
        out.append((n, c, h, w, k, r, s, st, pd))
    return out


RANDOM_LAYERS = _random_layers(16, 1356)


@pytest.mark.parametrize("spec", RANDOM_LAYERS, ids=[str(i) for i in range(len(RANDOM_LAYERS))])
def test_random_shapes_both_paths_match_oracle(spec):
    """Seeded random shapes: the runtime gradient and the plan (fused phases where
    the phase grids agree, windows over 3 x 3 through padded copies) against the
    oracle."""
    n, c, h, w, k, r, s, st, pd = spec
    dy, codes, _ = make(zlib.crc32(repr(spec).encode()), n, c, h, w, k, r, s, st, pd)
    want = oracle.conv2d_shift_backward_data(dy, codes, (n, c, h, w), r=r, s=s, stride=st, pad=pd)
    wph = ops.pack_shift_weights(codes)
    dx = ops.conv2d_shift_backward_data(to_dev(dy), to_dev(wph.view(np.int32)), (n, c, h, w), (r, s),
                                        st, pd).cpu().numpy()
    np.testing.assert_array_equal(dx, want, err_msg="runtime")
    plan = ops.JitConvBackwardData(wph, (n, c, h, w), (r, s), st, pd)
    say(f"backward random {spec}: {plan.segments} segments, {plan.splits} parts")
    dxp = plan(to_dev(dy)).cpu().numpy()
    plan.close()
    np.testing.assert_array_equal(dxp, want, err_msg="plan")
