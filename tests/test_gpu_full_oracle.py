"""Every output of every benchmark layer against the full oracle.

For each layer of the ResNet-18 (batch 32) and ResNet-50 (batch 128) workloads,
at the batch the benchmark times, both paths the benchmark runs -- the
weight-specialised plan made by ``ops.layer_plan`` (the benchmark's default)
and the runtime kernel (``ds_conv2d_shift`` / ``ds_linear_shift``) -- are
compared with the oracle on every output, bit for bit. The plan runs twice and
the two runs must agree as well.

On sampled outputs the float64 band of the paper's emulation (Section 4: the
float convolution with weights sign * 2^p) is checked too, in two forms:
|Y - Y_fp64| <= (number of accumulated terms) in units of 2^-F, and the exact
one-sided bound of the floor shift with the sign applied after the shift: a
positive term loses less than one unit, a negative term gains less than one,
so  -n_pos < Y - Y_exact < n_neg  (computed exactly in integers scaled by 2^14).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1905_13298_amd import ops
from paper_1905_13298_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

CASES = [(cfg, li, L.name) for cfg in (3, 4) for li, L in enumerate(W.config_layers(cfg))]


def say(*a):
    print(*a, flush=True)


def oracle_full(L, x, codes, bias):
    if L.kind == "linear":
        return oracle.linear_shift(x, codes, bias)
    return oracle.conv2d_shift(x, codes, bias, r=L.r, s=L.s, stride=L.stride, pad=L.pad)


def runtime_call(L, xt, wt, bt):
    if L.kind == "linear":
        return ops.linear_shift(xt, wt, bt)
    return ops.conv2d_shift(xt, wt, bt, (L.r, L.s), L.stride, L.pad)


def band_points(L, x, codes, bias, idx):
    """For flat output indices idx: (fp64 value, exact value * 2^14 as int64,
    positive and negative non-zero terms in the window) of the emulation."""
    shift = (codes & 15).astype(np.int64)
    nz = shift != 15
    neg = ((codes >> 4) & 1).astype(bool)
    sgn = np.where(neg, -1, 1) * nz
    e = np.where(nz, 14 - np.minimum(shift, 14), 0)          # 2^14 * 2^-shift = 2^e
    out = []
    if L.kind == "linear":
        for q in idx:
            b, k = divmod(int(q), L.k)
            xv = x[b].astype(np.int64)
            exact = int(np.sum(sgn[k] * (xv << e[k])))
            fp = float(np.sum(sgn[k] * np.ldexp(xv.astype(np.float64), -np.minimum(shift[k], 14))))
            npos, nneg = int(np.sum(nz[k] & ~neg[k])), int(np.sum(nz[k] & neg[k]))
            bb = 0 if bias is None else int(bias[k])
            out.append((fp + bb, exact + (bb << 14), npos, nneg))
        return out
    C, R, S = L.c, L.r, L.s
    for q in idx:
        n, rest = divmod(int(q), L.k * L.oh * L.ow)
        k, p = divmod(rest, L.oh * L.ow)
        oh, ow = divmod(p, L.ow)
        ih = oh * L.stride - L.pad + np.arange(R)
        iw = ow * L.stride - L.pad + np.arange(S)
        vh, vw = (ih >= 0) & (ih < L.h), (iw >= 0) & (iw < L.w)
        win = np.zeros((C, R, S), np.int64)
        win[:, vh[:, None] & vw[None, :]] = x[n][:, ih[vh]][:, :, iw[vw]].reshape(C, -1)
        valid = np.broadcast_to((vh[:, None] & vw[None, :])[None], (C, R, S)).reshape(-1)
        xv = win.reshape(-1)
        sk, ek, shk = sgn[k] * valid, e[k], shift[k]
        exact = int(np.sum(sk * (xv << ek)))
        fp = float(np.sum(sk * np.ldexp(xv.astype(np.float64), -np.minimum(shk, 14))))
        npos = int(np.sum(nz[k] & ~neg[k] & valid))
        nneg = int(np.sum(nz[k] & neg[k] & valid))
        bb = 0 if bias is None else int(bias[k])
        out.append((fp + bb, exact + (bb << 14), npos, nneg))
    return out


def check_band(L, y_flat, x, codes, bias, idx):
    for q, (fp, exact14, npos, nneg) in zip(idx, band_points(L, x, codes, bias, idx)):
        yq = int(y_flat[q])
        assert abs(yq - fp) <= L.crs, (q, yq, fp)
        d14 = (yq << 14) - exact14                 # (Y - exact) * 2^14
        lo_ok = d14 > -(npos << 14) if npos else d14 >= 0
        hi_ok = d14 < (nneg << 14) if nneg else d14 <= 0
        assert lo_ok and hi_ok, (q, yq, d14 / 16384.0, npos, nneg)


@pytest.mark.parametrize("cfg,li,name", CASES, ids=[f"{W.CONFIG_NAMES[c]}-{n}" for c, _, n in CASES])
def test_every_output_at_benchmark_batch(cfg, li, name):
    L = W.config_layers(cfg)[li]
    say(f"{W.CONFIG_NAMES[cfg]} layer {li} {name} batch {L.n}: oracle on {oracle.max_threads()} threads")
    x, codes, bias = W.gen_layer(L, W.CONFIG_SEEDS[cfg], li)
    want = oracle_full(L, x, codes, bias).reshape(-1)
    wp = ops.pack_shift_weights(codes)
    xt = torch.from_numpy(x).to(DEV)
    wt = torch.from_numpy(wp.view(np.int32)).to(DEV)
    bt = None if bias is None else torch.from_numpy(bias).to(DEV)

    plan = ops.layer_plan(L, wp, bias, device=DEV)
    y1 = ops.run_layer_plan(plan, L, xt).cpu().numpy().reshape(-1)
    y2 = ops.run_layer_plan(plan, L, xt).cpu().numpy().reshape(-1)
    plan.close()
    bad = np.flatnonzero(y1 != want)
    assert bad.size == 0, f"plan: {bad.size} of {want.size} outputs differ, first at {bad[:5]}"
    assert np.array_equal(y1, y2), "plan: two runs differ"

    yr = runtime_call(L, xt, wt, bt).cpu().numpy().reshape(-1)
    bad = np.flatnonzero(yr != want)
    assert bad.size == 0, f"runtime kernel: {bad.size} of {want.size} outputs differ, first at {bad[:5]}"

    rng = np.random.default_rng([cfg, li, 9])
    idx = np.unique(np.concatenate([rng.choice(want.size, 300, replace=False), [0, want.size - 1]]))
    check_band(L, y1, x, codes, bias, idx)


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_fp64_band_single_layer_configs_every_output(cfg):
    """The float64 band on every output of the three single-layer workloads, on both
    paths (their every output also equals the oracle's: test_gpu_parity, test_gpu_jit)."""
    import torch.nn.functional as F
    (L,) = W.config_layers(cfg)
    x, codes, bias = W.gen_layer(L, W.CONFIG_SEEDS[cfg], 0)
    wp = ops.pack_shift_weights(codes)
    xt = torch.from_numpy(x).to(DEV)
    bt = None if bias is None else torch.from_numpy(bias).to(DEV)
    plan = ops.layer_plan(L, wp, bias, device=DEV)
    ys = {"plan": ops.run_layer_plan(plan, L, xt).cpu().numpy(),
          "runtime": runtime_call(L, xt, torch.from_numpy(wp.view(np.int32)).to(DEV), bt).cpu().numpy()}
    plan.close()
    shift = (codes & 15).astype(np.int64)
    wf = np.where(shift == 15, 0.0, np.ldexp(1.0, -np.minimum(shift, 14)))
    wf = np.where((codes >> 4) & 1, -wf, wf)
    if L.kind == "linear":
        ref = x.astype(np.float64) @ wf.T
    else:
        ref = F.conv2d(torch.from_numpy(x.astype(np.float64)),
                       torch.from_numpy(wf.reshape(L.k, L.c, L.r, L.s)),
                       stride=L.stride, padding=L.pad).numpy()
    if bias is not None:
        ref = ref + (bias.reshape(1, -1) if L.kind == "linear" else bias.reshape(1, -1, 1, 1))
    for name, y in ys.items():
        d = y.astype(np.float64) - ref
        assert np.all(np.abs(d) <= L.crs), (cfg, name, float(np.abs(d).max()))
    # The exact one-sided bound on a sample of outputs.
    rng = np.random.default_rng(100 + cfg)
    total = int(np.prod(L.y_shape))
    idx = np.unique(np.concatenate([rng.choice(total, min(total, 500), replace=False), [0, total - 1]]))
    check_band(L, ys["plan"].reshape(-1), x, codes, bias, idx)
