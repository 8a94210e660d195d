"""The cost model behind JitConv.preferred (host arithmetic only): the plan and
runtime-kernel estimates for layouts the planner produces on the benchmark
shapes, against the durations measured on MI355X that the model was fitted to,
and the choice it makes."""
import pytest

from paper_1905_13298_amd import ops


def fake_plan(n, c, h, w, k, r, s, oh, ow, code_bytes, segments, splits, channels, wsplit, tiles,
              transposed=False):
    p = object.__new__(ops.JitConv)
    p.k = k
    p.crs = c * r * s
    p.out_pixels, p.out_channels = n * oh * ow, k
    p.sac = p.out_pixels * k * p.crs
    p.linear = h == w == r == s == 1
    p.code_bytes, p.segments, p.splits = code_bytes, segments, splits
    p.channels, p.wsplit, p.pixel_tiles = channels, wsplit, tiles
    p.pixel_groups = 1 if transposed else (4 // wsplit if wsplit <= 4 else 1)
    p.transposed = transposed
    return p


# (shape, layout as the planner makes it, measured plan us, measured runtime us),
# replays of HIP graphs on MI355X (the runtime convolution: eager calls)
CASES = [
    # 128 -> 128, 3 x 3 at 28 x 28, batch 1: 16-channel segments, wave split 8, 2 parts
    ((1, 128, 28, 28, 128, 3, 3, 28, 28), (868000, 16, 2, 16, 8, 13), 8.6, 42.1),
    # 256 -> 128 at batch 8: 16-channel segments, wave split 8; small-batch runtime kernel
    ((8, 256, 1, 1, 128, 1, 1, 1, 1), (257528, 8, 1, 16, 8, 1), 4.2, 4.46),
    # 512 -> 1000 at batch 32: 16-channel segments, wave split 4; small-batch runtime kernel
    ((32, 512, 1, 1, 1000, 1, 1, 1, 1), (3273484, 63, 1, 16, 4, 1), 10.2, 6.53),
    # 25088 -> 4096 at batch 1: split in 4; small-batch runtime kernel
    ((1, 25088, 1, 1, 4096, 1, 1, 1, 1), (450e6, 256, 4, 64, 4, 1), 344.3, 41.2),
    # On x^T (batch >= 64): 4096 -> 4096 at batch 256, 64-channel segments, wave
    # split 16, 4 tiles of 64 rows
    ((256, 4096, 1, 1, 4096, 1, 1, 1, 1), (74.3e6, 64, 1, 64, 16, 4, True), 108.7, 346.9),
    # 2048 -> 1000 at batch 128: 32-channel segments, wave split 16, 4 parts
    ((128, 2048, 1, 1, 1000, 1, 1, 1, 1), (10.7e6, 128, 4, 32, 16, 2, True), 17.0, 35.7),
    # 1024 -> 1024 at batch 64: the same layout
    ((64, 1024, 1, 1, 1024, 1, 1, 1, 1), (5.95e6, 128, 4, 32, 16, 1, True), 11.9, 13.7),
    # 512 -> 512 at batch 128: wave split 8, 4 parts; small-batch runtime kernel
    ((128, 512, 1, 1, 512, 1, 1, 1, 1), (1.5e6, 64, 4, 32, 8, 2, True), 10.3, 8.44),
]


@pytest.mark.parametrize("case", CASES, ids=["conv_n1", "linear_b8", "fc_b32", "fc6_b1", "fc_b256_xt",
                                              "fc_b128_xt", "fc_b64_xt", "fc_b128_small_xt"])
def test_model_tracks_measured_durations_and_picks_the_faster_path(case):
    shape, layout, plan_us, rt_us = case
    p = fake_plan(*shape, *layout)
    est, rt = p.estimate_us(), p.runtime_estimate_us()
    assert 0.7 * plan_us <= est <= 1.35 * plan_us, (est, plan_us)
    assert 0.7 * rt_us <= rt <= 1.35 * rt_us, (rt, rt_us)
    assert p.preferred == (plan_us < rt_us)


def test_model_prefers_the_runtime_kernel_for_much_code_and_little_work():
    # 4096 -> 4096 at batch 256 with 600 MB of code (a contrived plan, 8x what
    # the planner makes): the runtime kernel is estimated faster
    p = fake_plan(256, 4096, 1, 1, 4096, 1, 1, 1, 1, 600e6, 64, 1, 64, 4, 4, True)
    assert p.estimate_us() > p.runtime_estimate_us() and not p.preferred
