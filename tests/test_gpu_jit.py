"""GPU parity of the weight-specialised ConvShift plans (``ds_jit_conv_*``).

Each plan's output is compared with the oracle element by element on seeded
inputs: edge shapes (ragged channels, pixels and output channels; strides,
padding, rectangular windows; LinearShift as 1 x 1 on 1 x 1 images), each with
the reduction whole, split automatically and split by force (the split-K path
adds partial sums atomically and runs the epilogue as a pass of its own); the
fused epilogue (affine map, residual, ReLU) against the oracle's; segments of
16, 32 and 64 channels with wave splits up to 16; every block order of the grid;
the single-
layer workloads in full; and every ResNet-50 convolution (the 7 x 7 stem through
a padded copy of x) at batch 128 in full against the production kernel, plus
sampled outputs against the oracle.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops
from paper_1905_13298_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def rand_case(seed, n, c, h, w, k, r, s, small_x=False):
    rng = np.random.default_rng(seed)
    sign = rng.integers(0, 2, (k, c * r * s))
    shift = rng.integers(0, 16, (k, c * r * s))
    codes = (sign << 4 | shift).astype(np.uint8)
    lim = 2 ** 18 if small_x else 2 ** 31
    x = rng.integers(-lim, lim, (n, c, h, w), dtype=np.int64).astype(np.int32)
    bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
    return codes, x, bias, rng


EDGE = [
    # name, n, c, h, w, k, r, s, stride, pad
    ("ragged_k_c_pix", 3, 13, 9, 11, 37, 3, 3, 1, 1),
    ("1x1_s2", 3, 20, 15, 15, 33, 1, 1, 2, 0),
    ("1x1_s1_odd", 2, 9, 7, 5, 70, 1, 1, 1, 0),
    ("1x1_pad", 1, 5, 6, 6, 9, 1, 1, 1, 1),
    ("3x3_s2_odd", 2, 11, 13, 9, 17, 3, 3, 2, 1),
    ("3x3_s3_pad2", 1, 6, 17, 17, 8, 3, 3, 3, 2),
    ("rect_2x3", 2, 5, 10, 12, 6, 2, 3, 1, 1),
    ("7x7_images", 5, 16, 7, 7, 40, 3, 3, 1, 1),
    ("linear_like", 70, 300, 1, 1, 130, 1, 1, 1, 0),
    ("tiny", 1, 1, 1, 1, 1, 1, 1, 1, 0),
    ("big_c_small_k", 1, 300, 6, 6, 3, 3, 3, 1, 1),
    ("many_tiles", 4, 64, 20, 20, 128, 3, 3, 1, 1),
    # windows over 3 x 3 read a zero-padded copy of x
    ("7x7_s2_stem_like", 2, 3, 23, 21, 70, 7, 7, 2, 3),
    ("5x5_pad2", 2, 9, 12, 10, 40, 5, 5, 1, 2),
    ("4x6_s3_cropped", 1, 6, 14, 17, 20, 4, 6, 3, 0),
    ("1x7_pad3", 2, 5, 9, 16, 33, 1, 7, 1, 3),
]


@pytest.mark.parametrize("splits", [1, 0, 3])
@pytest.mark.parametrize("spec", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes_match_oracle(spec, splits):
    name, n, c, h, w, k, r, s, st, pd = spec
    codes, x, bias, _ = rand_case(zlib.crc32(name.encode()) + splits, n, c, h, w, k, r, s)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, (r, s), st, pd, bias=bias,
                       splits=splits)
    say(f"jit {name} splits={splits} -> {plan.splits} parts, {plan.segments} segments, "
        f"{plan.code_bytes} code bytes")
    y = plan(to_dev(x)).cpu().numpy()
    want = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    bad = np.flatnonzero(y.ravel() != want.ravel())
    assert bad.size == 0, f"{bad.size} of {want.size} outputs differ, first at {bad[:5]}"


LAYOUTS = [(16, 4), (16, 8), (16, 16), (32, 16), (64, 8), (64, 16), (32, 2)]
LAYOUT_SHAPES = ["ragged_k_c_pix", "1x1_s2", "linear_like", "7x7_s2_stem_like", "big_c_small_k",
                 "tiny", "many_tiles"]


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("layout", LAYOUTS, ids=[f"tn{a}_ws{b}" for a, b in LAYOUTS])
@pytest.mark.parametrize("name", LAYOUT_SHAPES)
def test_segment_widths_and_wave_splits_match_oracle(name, layout, splits, knob):
    """Segments of 16, 32 or 64 output channels with wave splits up to 16 (workgroups
    of up to 1024 threads meeting in LDS), whole and split, against the oracle."""
    spec = next(e for e in EDGE if e[0] == name)
    _, n, c, h, w, k, r, s, st, pd = spec
    tn, ws = layout
    knob("DS_JIT_TN", tn)
    knob("DS_JIT_WSPLIT", ws)
    codes, x, bias, _ = rand_case(zlib.crc32(repr((spec, layout, splits)).encode()), n, c, h, w, k, r, s)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, (r, s), st, pd, bias=bias, splits=splits)
    say(f"jit layout tn{tn} ws{ws} {name} splits={splits}: {plan.splits} parts, {plan.segments} segments")
    y = plan(to_dev(x)).cpu().numpy()
    plan.close()
    want = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    bad = np.flatnonzero(y.ravel() != want.ravel())
    assert bad.size == 0, f"{bad.size} of {want.size} outputs differ, first at {bad[:5]}"


@pytest.mark.parametrize("layout", [(16, 16), (32, 8), (16, 4)])
def test_epilogue_in_narrow_segments_matches_oracle(layout, knob):
    """The fused epilogue (affine map, residual, ReLU) when each of up to 16 waves
    finishes one or a few channels of a 16- or 32-channel segment."""
    tn, ws = layout
    knob("DS_JIT_TN", tn)
    knob("DS_JIT_WSPLIT", ws)
    n, c, h, w, k, r, s, st, pd = 2, 40, 11, 11, 70, 3, 3, 1, 1
    codes, x, bias, rng = rand_case(zlib.crc32(repr(layout).encode()), n, c, h, w, k, r, s, small_x=True)
    mul = rng.integers(-(2 ** 17), 2 ** 17, k).astype(np.int32)
    add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    res = rng.integers(-(2 ** 24), 2 ** 24, (n, k, h, w)).astype(np.int32)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, 3, st, pd, bias=bias, mul=mul, add=add,
                       mul_shift=16, residual=True, relu=True, splits=1)
    say(f"jit epilogue tn{tn} ws{ws}")
    y = plan(to_dev(x), residual=to_dev(res)).cpu().numpy()
    plan.close()
    conv = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    np.testing.assert_array_equal(y, oracle.epilogue(conv, mul, add, 16, residual=res, relu=True))


@pytest.mark.parametrize("splits", [1, 2])
@pytest.mark.parametrize("parts", ["mul", "mul_add_relu", "residual_relu", "all", "relu"])
def test_epilogue_matches_oracle(parts, splits):
    n, c, h, w, k, r, s, st, pd = 2, 24, 11, 11, 70, 3, 3, 1, 1
    codes, x, bias, rng = rand_case(zlib.crc32(parts.encode()) + splits, n, c, h, w, k, r, s,
                                    small_x=True)
    mul = add = res = None
    if "mul" in parts or parts == "all":
        mul = rng.integers(-(2 ** 17), 2 ** 17, k).astype(np.int32)
    if "add" in parts or parts == "all":
        add = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    if "residual" in parts or parts == "all":
        res = rng.integers(-(2 ** 24), 2 ** 24, (n, k, h, w)).astype(np.int32)
    relu = "relu" in parts or parts == "all"
    say(f"jit epilogue {parts} splits={splits}")
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, 3, st, pd, bias=bias, mul=mul,
                       add=add, mul_shift=16, residual=res is not None, relu=relu, splits=splits)
    y = plan(to_dev(x), residual=to_dev(res)).cpu().numpy()
    conv = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    want = oracle.epilogue(conv, mul, add, 16, residual=res, relu=relu)
    np.testing.assert_array_equal(y, want)


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_single_layer_configs_exact(cfg):
    (layer,) = W.config_layers(cfg)
    x, codes, bias = W.gen_layer(layer, W.CONFIG_SEEDS[cfg], 0)
    lin = layer.kind == "linear"
    shape = (layer.n, layer.c, 1, 1) if lin else x.shape
    say(f"jit {W.CONFIG_NAMES[cfg]} {layer.name}")
    plan = ops.JitConv(ops.pack_shift_weights(codes), shape, (1, 1) if lin else (layer.r, layer.s),
                       1 if lin else layer.stride, 0 if lin else layer.pad, bias=bias)
    y = plan(to_dev(x.reshape(shape))).cpu().numpy()
    if lin:
        want = oracle.linear_shift(x, codes, bias)
        y = y.reshape(want.shape)
    else:
        want = oracle.conv2d_shift(x, codes, bias, r=layer.r, s=layer.s, stride=layer.stride,
                                   pad=layer.pad)
    bad = np.flatnonzero(y.ravel() != want.ravel())
    assert bad.size == 0, f"{bad.size} of {want.size} outputs differ, first at {bad[:5]}"


def test_plan_is_reusable_and_checks_its_arguments():
    n, c, h, w, k = 2, 10, 6, 6, 8
    codes, x, bias, rng = rand_case(5, n, c, h, w, k, 3, 3)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, 3, 1, 1, bias=bias)
    for i in range(3):
        xi = rng.integers(-(2 ** 31), 2 ** 31, x.shape, dtype=np.int64).astype(np.int32)
        y = plan(to_dev(xi)).cpu().numpy()
        np.testing.assert_array_equal(y, oracle.conv2d_shift(xi, codes, bias, r=3, stride=1, pad=1))
    xd = to_dev(x)
    with pytest.raises(ops.DeepShiftError, match="residual must be NULL"):
        plan(xd, residual=torch.zeros((n, k, h, w), dtype=torch.int32, device=DEV))
    with pytest.raises(ops.DeepShiftError, match="overlaps"):
        plan(xd, out=xd.view(-1)[: n * k * h * w].view(n, k, h, w))
    rplan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, 3, 1, 1, residual=True)
    with pytest.raises(ops.DeepShiftError, match="residual must not be NULL"):
        rplan(xd)
    res = torch.zeros((n, k, h, w), dtype=torch.int32, device=DEV)
    with pytest.raises(ops.DeepShiftError, match="overlaps residual"):
        rplan(xd, residual=res, out=res)
    plan.close()
    rplan.close()


def test_plans_replay_in_a_captured_graph():
    """Plans allocate nothing and launch only kernels when run (the padding, fill
    and epilogue passes included), so a stream capture of several plans replays:
    three replays, with the outputs overwritten eagerly between them, each equal
    to the eager result, itself equal to the oracle."""
    rng = np.random.default_rng(77)
    cases = [  # n, c, h, w, k, r, s, stride, pad, splits: padded 5x5, wave split, split-K,
        # LinearShifts on x^T (transposing passes; the first pass also fills y^T when split)
        (2, 3, 15, 13, 40, 5, 5, 2, 2, 0),
        (2, 40, 9, 9, 70, 3, 3, 1, 1, 0),
        (3, 300, 6, 6, 9, 1, 1, 1, 0, 3),
        (70, 300, 1, 1, 130, 1, 1, 1, 0, 1),
        (64, 200, 1, 1, 90, 1, 1, 1, 0, 3),
    ]
    runs, wants = [], []
    for (n, c, h, w, k, r, s, st, pd, sp) in cases:
        codes = random_codes_like(rng, k, c * r * s)
        x = rng.integers(-(2 ** 31), 2 ** 31, (n, c, h, w), dtype=np.int64).astype(np.int32)
        bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
        plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, (r, s), st, pd, bias=bias,
                           splits=sp)
        xd = to_dev(x)
        y = torch.empty(plan.y_shape, dtype=torch.int32, device=DEV)
        runs.append((plan, xd, y))
        wants.append(oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd))
    for plan, xd, y in runs:
        plan(xd, out=y)
    torch.cuda.synchronize()
    for (_, _, y), want in zip(runs, wants):
        np.testing.assert_array_equal(y.cpu().numpy(), want)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for plan, xd, y in runs:
            plan(xd, out=y)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, capture_error_mode="thread_local"):
        for plan, xd, y in runs:
            plan(xd, out=y)
    for rep in range(3):
        for _, _, y in runs:
            y.fill_(0x5A5A5A5A)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for (_, _, y), want in zip(runs, wants):
            np.testing.assert_array_equal(y.cpu().numpy(), want, err_msg=f"replay {rep}")
    say(f"graph of {len(runs)} plans: 3 replays equal the oracle")
    del graph
    for plan, _, _ in runs:
        plan.close()


def random_codes_like(rng, k, cols, zero_frac=0.2):
    sign = rng.integers(0, 2, (k, cols))
    shift = rng.integers(0, 15, (k, cols))
    shift[rng.random((k, cols)) < zero_frac] = 15
    return (sign << 4 | shift).astype(np.uint8)


def _random_layers(count, seed):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        n, c, k = int(rng.integers(1, 5)), int(rng.integers(1, 200)), int(rng.integers(1, 200))
        r, s = int(rng.integers(1, 8)), int(rng.integers(1, 8))
        st, pd = int(rng.integers(1, 4)), int(rng.integers(0, 4))
        h, w = int(rng.integers(1, 30)), int(rng.integers(1, 30))
        if h + 2 * pd < r or w + 2 * pd < s:
            continue
        out.append((n, c, h, w, k, r, s, st, pd))
    return out


ORDER_CASES = [
    # pixel tiles not a multiple of 8 (a partial last row of tiles), fewer than 8,
    # and a strided 1 x 1 layer
    ("ragged_rows", 2, 40, 28, 29, 130, 3, 3, 1, 1),
    ("point_s2", 4, 64, 30, 30, 96, 1, 1, 2, 0),
    ("many_tiles", 8, 32, 20, 20, 64, 3, 3, 1, 1),
    ("few_tiles", 1, 24, 9, 9, 200, 3, 3, 1, 1),
]


@pytest.mark.parametrize("spec", ORDER_CASES, ids=[e[0] for e in ORDER_CASES])
def test_block_orders_match_oracle(spec, knob):
    """Every block order (grouped, tile-major, tile-major with a tile's workgroups
    on one XCD) maps the grid onto all (tile, segment) pairs once: each gives the
    oracle's output."""
    _, n, c, h, w, k, r, s, st, pd = spec
    codes, x, bias, _ = rand_case(zlib.crc32(repr(spec).encode()), n, c, h, w, k, r, s)
    want = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, (r, s), st, pd, bias=bias)
    xd = to_dev(x)
    for order in (0, 1, 2):
        knob("DS_JIT_ORDER", order)
        say(f"jit order {order} {spec[0]}: {plan.segments} segments, {plan.pixel_tiles} tiles")
        y = plan(xd).cpu().numpy()
        bad = np.flatnonzero(y.ravel() != want.ravel())
        assert bad.size == 0, f"order {order}: {bad.size} of {want.size} outputs differ, first at {bad[:5]}"
    plan.close()


RANDOM_LAYERS = _random_layers(16, 355)


@pytest.mark.parametrize("spec", RANDOM_LAYERS, ids=[str(i) for i in range(len(RANDOM_LAYERS))])
def test_random_shapes_match_oracle(spec):
    """Seeded random shapes (windows up to 7 x 7, strides up to 3, padding up to 3)
    with the planner's own choices of wave split and split-K."""
    n, c, h, w, k, r, s, st, pd = spec
    codes, x, bias, _ = rand_case(zlib.crc32(repr(spec).encode()), n, c, h, w, k, r, s)
    plan = ops.JitConv(ops.pack_shift_weights(codes), x.shape, (r, s), st, pd, bias=bias)
    say(f"jit random {spec}: {plan.splits} parts, {plan.segments} segments")
    y = plan(to_dev(x)).cpu().numpy()
    plan.close()
    want = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    bad = np.flatnonzero(y.ravel() != want.ravel())
    assert bad.size == 0, f"{bad.size} of {want.size} outputs differ, first at {bad[:5]}"


MUL_PLAN_CASES = [
    # name, n, c, h, w, k, r, s, stride, pad, splits
    ("window", 2, 40, 9, 9, 70, 3, 3, 1, 1, 0),
    ("strided_split", 3, 37, 14, 14, 64, 3, 3, 2, 1, 3),
    ("pointwise", 2, 64, 28, 28, 256, 1, 1, 1, 0, 0),
    ("stem_padded", 1, 3, 35, 35, 64, 7, 7, 2, 3, 0),
    ("linear", 8, 256, 1, 1, 128, 1, 1, 1, 0, 0),
]


@pytest.mark.parametrize("spec", MUL_PLAN_CASES, ids=[e[0] for e in MUL_PLAN_CASES])
def test_multiplication_plans_match_oracle(spec):
    """Multiplication plans (the comparison operator in the plans' tiling) against
    the oracle's 24-bit product, with inline-constant, literal and zero weights and
    inputs beyond 24 bits."""
    _, n, c, h, w, k, r, s, st, pd, splits = spec
    rng = np.random.default_rng(zlib.crc32(repr(spec).encode()))
    wt = rng.integers(-(2 ** 31), 2 ** 31, (k, c * r * s), dtype=np.int64).astype(np.int32)
    small = rng.random(wt.shape) < 0.3
    wt[small] = rng.integers(-16, 65, int(small.sum()))
    wt[rng.random(wt.shape) < 0.2] = 0
    x = rng.integers(-(2 ** 31), 2 ** 31, (n, c, h, w), dtype=np.int64).astype(np.int32)
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    plan = ops.JitConvMul(wt, x.shape, (r, s), st, pd, bias=bias, splits=splits)
    say(f"mul plan {spec[0]}: {plan.splits} parts, {plan.code_bytes} code bytes")
    y = plan(to_dev(x)).cpu().numpy()
    plan.close()
    np.testing.assert_array_equal(y, oracle.conv2d_mul24(x, wt, bias, r=r, s=s, stride=st, pad=pd))


def _graph_us(fn, reps=10, outer=5):
    fn()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            for _ in range(reps):
                fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(outer):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (reps * outer) * 1000.0


@pytest.mark.parametrize("n,c,k", [(256, 4096, 4096), (1, 25088, 4096)], ids=["fc_b256", "fc6_b1"])
def test_cost_model_choice_matches_measurement(n, c, k):
    """JitConv.preferred against both paths timed (as graph replays) on two
    LinearShift shapes whose measured gap is wide (2x and 7x on MI355X): the
    path the model picks must be the faster one by at least 1.3x, and both paths
    must give the oracle's result on sampled outputs."""
    rng = np.random.default_rng(c)
    x = rng.integers(0, 2 ** 17, (n, c)).astype(np.int32)
    codes = W.random_codes(rng, (k, c), zero_frac=0.1)
    bias = rng.integers(-(2 ** 16), 2 ** 16, k).astype(np.int32)
    wp = ops.pack_shift_weights(codes)
    xt, wt, bt = to_dev(x), to_dev(wp.view(np.int32)), to_dev(bias)
    plan = ops.JitConv(wp, (n, c, 1, 1), 1, 1, 0, bias=bias)
    y_rt = torch.empty((n, k), dtype=torch.int32, device=DEV)
    y_pl = torch.empty((n, k, 1, 1), dtype=torch.int32, device=DEV)
    t_rt = _graph_us(lambda: ops.linear_shift(xt, wt, bt, out=y_rt))
    t_pl = _graph_us(lambda: plan(xt.view(n, c, 1, 1), out=y_pl))
    say(f"cost model {n}x{c}->{k}: plan {t_pl:.1f} us (model {plan.estimate_us():.1f}), "
        f"runtime {t_rt:.1f} us (model {plan.runtime_estimate_us():.1f}), preferred {plan.preferred}")
    assert torch.equal(y_rt, y_pl.view(n, k))
    idx = rng.integers(0, n * k, 200)
    got = y_rt.cpu().numpy().ravel()[idx]
    want = oracle.linear_shift_points(x, codes, bias, idx)
    np.testing.assert_array_equal(got, want)
    plan_faster = t_pl * 1.3 < t_rt
    runtime_faster = t_rt * 1.3 < t_pl
    assert plan_faster or runtime_faster, "the two paths are too close to judge"
    assert plan.preferred == plan_faster
    plan.close()
