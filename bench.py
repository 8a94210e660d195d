"""Benchmark of the DeepShift shift operators on one MI355X.

A step is one pass of every layer of the workload (each layer's ConvShift or
LinearShift call on its own seeded input, all inputs resident in HBM).
Two paths compute the same outputs bit for bit (checked before timing):
  jit      (default) a weight-specialised plan per layer, its code generated
           at setup from the fixed weights (Section 6's run-time compilation);
           a layer whose plan is not preferred (JitConv.preferred: a cost
           model of both paths, in the per-layer JSON) runs the runtime kernel
  runtime  ds_conv2d_shift / ds_linear_shift with the packed weights as data
Prints ONE JSON line:
  value       whole-step throughput in G shift-accumulates/s (dense SAC =
              output elements x reduction terms, zero weights included)
  roofline    the dominant kernel against the int32 VALU roofline: the runtime
              kernel at 2 VALU instructions per dense shift-accumulate (one of
              them three-operand, 64 lanes per CU per clock); the generated
              kernel at one two-operand add/sub per non-zero weight term (128
              lanes per CU per clock)
  runtime_weights  the runtime path timed on the same inputs (path jit)
  cpu_baseline the oracle on the host cores, on a prefix (small batch) of
              the same seeded inputs
  mul_comparison  the multiplication-based comparison on the same layers, at
              the tiling of each shift path: int32 and 24-bit multiply-adds in
              the runtime kernel's tiling, 24-bit multiply-adds baked into
              plans like the shifts

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload resnet50]
                       [--path jit|runtime]
K defaults to 24 for a network and 640 for a single layer (whose steps last
microseconds), W to 2.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOADS = {"linear_small": 0, "conv_single": 1, "linear_fc6": 2, "resnet18": 3, "resnet50": 4}
# A plan that is almost only VOP2 adds and subtracts (workloads.VALU_PROBE): its rate,
# and its SQ counters under rocprofv3, measure the issue rate of generated code.
PROBE_WORKLOADS = {"valu_probe": 99}
# A layer where the plans' cost model prefers the runtime kernel: VGG16's fc6
# (25088 -> 4096) at batch 1, about 450 MB of generated code for one row. With
# --time-rejected the rejected plan is timed too, to check the model's choice.
MODEL_WORKLOADS = {"linear_25088_b1": 98}
# The step upstream of the operators: float weights -> packed codes (DeepShift-Q)
# and the float input batch -> fixed point, for every layer of ResNet-50 at N = 128.
CONVERT_WORKLOADS = {"convert_resnet50": 4}
# Chained inference: a ResNet-18 forward pass with shift convolutions (batch
# normalisation, residual and ReLU fused into each convolution), N = 32.
NETWORK_WORKLOADS = {"resnet18_infer": 32}
# Input gradients (the data half of the backward pass) of every layer of a
# workload but the stem (the images need no gradient), on signed output gradients.
BACKWARD_WORKLOADS = {"resnet50_bwd_data": 4, "resnet18_bwd_data": 3}

# MI355X: 256 CUs of 4 SIMDs at 2.4 GHz; a wave64 VALU instruction occupies a
# SIMD for 4 clocks, i.e. 64 int32 lane-ops per CU per clock (39.32 T/s). The
# SIMDs also issue two-operand (VOP2) instructions such as v_add_u32 /
# v_sub_u32 / v_ashrrev_i32 two at a time from different waves (the counter
# SQ_ACTIVE_INST_VALU2): a register-only probe issued 0.39-0.45 such
# instructions per SIMD per clock against 0.24 for three-operand ones, and the
# generated plan code reached 0.355 per SIMD per clock with 90 % of them in pairs
# (profiles/valu_issue_rates.md). The plans are therefore rated against 128 lane-ops per
# CU per clock (78.64 T/s), and also reported against 39.32 T/s.
CUS, LANES_PER_CU, CLOCK_GHZ = 256, 64, 2.4
INT32_OPS_PEAK_T = CUS * LANES_PER_CU * CLOCK_GHZ / 1000.0        # 39.32 T int32 ops/s (VOP3)
VOP2_OPS_PEAK_T = 2 * INT32_OPS_PEAK_T                              # 78.64 T int32 ops/s (VOP2)
SAC_PEAK_T = INT32_OPS_PEAK_T / 2.0                                  # 19.66 T SAC/s
HBM_PEAK_GBS = 8000.0


def kernel_variant(layer) -> str:
    """The kernel the library runs for a layer, as the library itself names it."""
    from paper_1905_13298_amd import ops
    if layer.kind == "linear":
        return ops.describe_conv2d(layer.n, layer.c, 1, 1, layer.k, 1)
    return ops.describe_conv2d(layer.n, layer.c, layer.h, layer.w, layer.k, (layer.r, layer.s),
                               layer.stride, layer.pad)


def algorithmic_bytes(layer, act_bits: int = 32) -> int:
    """Bytes a call must move at least: x (act_bits per element), y, packed weights
    (ceil(CRS/6) words per row), bias."""
    wpr = (layer.crs + 5) // 6
    b = act_bits // 8 * int(np.prod(layer.x_shape)) + 4 * int(np.prod(layer.y_shape)) + 4 * layer.k * wpr
    return b + (4 * layer.k if layer.bias else 0)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: 640 for a single layer, whose step lasts microseconds, "
                         "24 for a network, so that graph launches are a small part of the timed region)")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="resnet50", choices=sorted(WORKLOADS) + sorted(CONVERT_WORKLOADS) + sorted(NETWORK_WORKLOADS)
                    + sorted(BACKWARD_WORKLOADS) + sorted(PROBE_WORKLOADS) + sorted(MODEL_WORKLOADS))
    ap.add_argument("--eager", action="store_true",
                    help="path jit: time eager calls instead of replays of a HIP graph of the step")
    ap.add_argument("--time-rejected", action="store_true",
                    help="with --path jit, also time the plans the cost model rejects (per-layer JSON)")
    ap.add_argument("--cpu-batch", type=int, default=None,
                    help="batch of the oracle sample (default: sized for ~10-30 s)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time the CPU baseline aims for (whole passes over its sample)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-mul", action="store_true")
    ap.add_argument("--layers-out", default=None, help="write per-layer timings (JSON) here")
    ap.add_argument("--copy-only", type=int, default=0, metavar="BYTES",
                    help="only run a device-to-device copy of BYTES (HBM counter calibration)")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("COPY_FETCH", "COPY_WRITE", "FETCH", "WRITE"),
                    help="turn rocprofv3 --pmc CSV directories into the HBM traffic record")
    ap.add_argument("--sq-summary", metavar="DIR",
                    help="summarise a rocprofv3 --pmc run with SQ instruction counters per kernel")
    ap.add_argument("--pmc-copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--pmc-out", default=None,
                    help="traffic record to write (default: the committed one of --path)")
    ap.add_argument("--path", default="jit", choices=["jit", "runtime"],
                    help="jit: weight-specialised plans made at setup (layers they do not cover "
                         "run the runtime kernel); runtime: ds_conv2d_shift / ds_linear_shift")
    ap.add_argument("--no-runtime", action="store_true",
                    help="with --path jit, skip timing the runtime-weights path as well")
    ap.add_argument("--act-bits", type=int, default=32, choices=[32, 16, 8],
                    help="activation width of the layer workloads: 32 (int32, F=16), or the lower "
                         "bit-widths 16 (int16 3.13) and 8 (int8 3.5), on the plan path")
    return ap.parse_args()


CSRC = os.path.join(ROOT, "paper_1905_13298_amd", "csrc")
# The generated weight-specialised kernel: one code object per plan with two
# entry points (up to 3 x 3 taps per element, 96 VGPRs; one tap, 80 VGPRs),
# accounted together under the first one's name.
JIT_KERNEL = "ds_jit_conv_template"
JIT_ENTRY_POINTS = ("ds_jit_conv_template", "ds_jit_conv_one_tap_template")


def is_jit_kernel(name: str) -> bool:
    return any(e in name for e in JIT_ENTRY_POINTS)

# Per kernel family: the sources its code comes from, and the committed HBM
# traffic record of its counters on the ResNet-50 workload.
FAMILIES = {
    "runtime": (["conv_kernels.hip"], os.path.join(ROOT, "profiles", "hbm_traffic_resnet50_n128.json")),
    "jit": (["jit.hip", "jit_template.hip"],
            os.path.join(ROOT, "profiles", "hbm_traffic_jit_resnet50_n128.json")),
}


def kernel_source_hash(family: str = "runtime") -> str:
    import hashlib
    h = hashlib.sha256()
    for src in FAMILIES[family][0]:
        with open(os.path.join(CSRC, src), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _pmc_rows(directory: str):
    """Per-dispatch counter sums from a rocprofv3 --pmc CSV directory."""
    import csv
    import glob
    (path,) = glob.glob(os.path.join(directory, "*counter_collection.csv"))
    rows = {}
    for r in csv.DictReader(open(path)):
        e = rows.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"], "ctr": {},
                                                     "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        e["ctr"][r["Counter_Name"]] = e["ctr"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [rows[k] for k in sorted(rows)]


MAIN_KERNELS = ("tiled_kernel", "conv_direct_kernel", "linear_rows_kernel") + JIT_ENTRY_POINTS


def _main_rows(rows, layers):
    """The last len(layers) dispatches of a main kernel: one per layer of the last step."""
    return [r for r in rows if any(m in r["name"] for m in MAIN_KERNELS)][-len(layers):]


def pmc_summary(copy_fetch, copy_write, fetch, write, copy_bytes, workload, path, out):
    """HBM traffic of the main (tiled, direct or generated) kernels from FETCH_SIZE/WRITE_SIZE
    runs (KiB per dispatch), each scaled by what the same counter reads for a plain copy of
    copy_bytes (the largest copy dispatch in the calibration runs)."""
    from paper_1905_13298_amd import workloads as W
    cf = max(r["ctr"]["FETCH_SIZE"] for r in _pmc_rows(copy_fetch) if "copyBuffer" in r["name"])
    cw = max(r["ctr"]["WRITE_SIZE"] for r in _pmc_rows(copy_write) if "copyBuffer" in r["name"])
    fetch_scale = copy_bytes / (cf * 1024.0)
    write_scale = copy_bytes / (cw * 1024.0)
    layers = W.config_layers(WORKLOADS[workload])
    f_rows = _main_rows(_pmc_rows(fetch), layers)
    w_rows = _main_rows(_pmc_rows(write), layers)
    per_kernel = {}
    for L, fr, wr in zip(layers, f_rows, w_rows):
        name = group_name(L, path, is_jit_kernel(fr["name"]))
        k = per_kernel.setdefault(name, {"launches": 0, "fetch_bytes": 0.0, "write_bytes": 0.0,
                                          "algorithmic_bytes": 0})
        k["launches"] += 1
        k["fetch_bytes"] += fr["ctr"]["FETCH_SIZE"] * 1024.0 * fetch_scale
        k["write_bytes"] += wr["ctr"]["WRITE_SIZE"] * 1024.0 * write_scale
        k["algorithmic_bytes"] += algorithmic_bytes(L)
    rec = {"workload": W.CONFIG_NAMES[WORKLOADS[workload]], "path": path,
           "kernel_source_sha256_16": kernel_source_hash(path),
           "copy_bytes": copy_bytes, "fetch_scale": round(fetch_scale, 4),
           "write_scale": round(write_scale, 4), "kernels": per_kernel}
    with open(out or FAMILIES[path][1], "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def sq_summary(directory, workload, path):
    """VALU evidence per kernel from one rocprofv3 --pmc run of the bench
    (one timed step, no warm-up) with SQ_WAVES SQ_INSTS_VALU SQ_INSTS_SALU
    SQ_INSTS_SMEM SQ_INSTS_LDS SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_INST_ANY and
    GRBM_GUI_ACTIVE: VALU instructions per shift-accumulate (dense and non-zero),
    VALU issue rate per SIMD per clock, and int32 lane-operations per second
    against the peak."""
    from paper_1905_13298_amd import workloads as W
    probe = workload in PROBE_WORKLOADS or workload in MODEL_WORKLOADS
    cfg = None if probe else WORKLOADS[workload]
    if probe:
        layers = [W.VALU_PROBE] if workload in PROBE_WORKLOADS else [W.LINEAR_25088_B1]
        seed = 99 if workload in PROBE_WORKLOADS else 98
    else:
        layers, seed = W.config_layers(cfg), W.CONFIG_SEEDS[cfg]
    rows = _main_rows(_pmc_rows(directory), layers)
    per = {}
    for li, (L, r) in enumerate(zip(layers, rows)):
        codes = W.gen_codes(L, seed, li)
        name = group_name(L, path, is_jit_kernel(r["name"]))
        k = per.setdefault(name, {"launches": 0, "sac": 0, "nz": 0.0, "ns": 0})
        k["launches"] += 1
        k["sac"] += L.sac
        k["nz"] += L.sac * float(np.mean((codes & 15) != 15))
        k["ns"] += r["ns"]
        for c, v in r["ctr"].items():
            k[c] = k.get(c, 0.0) + v
    out = {}
    for name, k in per.items():
        clk = k["GRBM_GUI_ACTIVE"] / 8.0          # GPU clocks, summed over the 8 XCDs
        valu = k["SQ_INSTS_VALU"]
        out[name] = {
            "launches": k["launches"], "ms": round(k["ns"] / 1e6, 3),
            "tsac_s": round(k["sac"] / k["ns"] / 1e3, 3),
            "clock_ghz": round(clk / k["ns"], 3),
            "valu_insts_per_sac": round(valu * 64 / k["sac"], 3),
            "valu_insts_per_nonzero_sac": round(valu * 64 / k["nz"], 3),
            "valu_issue_per_simd_clk": round(valu / (CUS * 4) / clk, 4),
            "int32_lane_ops_t": round(valu * 64 / k["ns"] / 1e3, 2),
            "frac_of_vop3_lane_rate": round(valu * 64 / k["ns"] / 1e3 / INT32_OPS_PEAK_T, 4),
            "frac_of_vop2_lane_rate": round(valu * 64 / k["ns"] / 1e3 / VOP2_OPS_PEAK_T, 4),
            "salu_per_valu": round(k["SQ_INSTS_SALU"] / valu, 3),
            "smem_per_valu": round(k["SQ_INSTS_SMEM"] / valu, 4),
            "lds_per_valu": round(k["SQ_INSTS_LDS"] / valu, 4),
            "wait_inst_any_per_wave_cycle": round(k["SQ_WAIT_INST_ANY"] / k["SQ_WAVE_CYCLES"], 3),
        }
    rec = {"workload": workload if probe else W.CONFIG_NAMES[cfg], "path": path,
           "kernel_source_sha256_16": kernel_source_hash(path), "kernels": out}
    print(json.dumps(rec, indent=1))


def measured_traffic(kernel: str, family: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter record, or None
    when there is none, it was taken on another workload, or the kernel source
    changed since it was taken."""
    try:
        rec = json.load(open(FAMILIES[family][1]))
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("kernel_source_sha256_16") != kernel_source_hash(family):
        return None
    k = rec["kernels"].get(kernel)
    if not k:
        return None
    return (k["fetch_bytes"] + k["write_bytes"]) / k["launches"]


def copy_only(nbytes: int) -> None:
    """A plain device-to-device copy of a known size, three times: what the HBM
    traffic counters read for it calibrates them."""
    import torch
    dev = torch.device("cuda:0")
    n = nbytes // 4
    src = torch.arange(n, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    print(json.dumps({"copy_bytes": 4 * n, "repeats": 3}), flush=True)


def bench_convert(args):
    """One step = DeepShift-Q conversion of every weight tensor of the network plus the
    fixed-point rounding of its input batch; HBM-bound, so reported in GB/s."""
    import torch
    from paper_1905_13298_amd import ops
    from paper_1905_13298_amd import workloads as W

    cfg = CONVERT_WORKLOADS[args.workload]
    layers = W.config_layers(cfg)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ws = [torch.from_numpy(W.gen_float_weights(L.k, L.crs, seed=1000 + i)).to(dev)
          for i, L in enumerate(layers)]
    outs = [torch.empty((L.k, ops.packed_row_words(L.crs)), dtype=torch.int32, device=dev)
            for L in layers]
    stem = layers[0]
    nx = int(np.prod(stem.x_shape))
    xf = torch.from_numpy(W.gen_float_acts(nx, seed=5)).to(dev)
    xq = torch.empty(nx, dtype=torch.int32, device=dev)
    w_bytes = sum(4 * w.numel() + 4 * o.numel() for w, o in zip(ws, outs))
    x_bytes = 8 * nx
    # One library call converts all weight tensors (launches of up to 64 tensors each).
    calls = [("quantize_q_many", ws, outs), ("to_fixed", xf, xq)]

    def run(call):
        kind, a, o = call
        if kind == "quantize_q_many":
            ops.quantize_shift_weights_q_many(a, outs=o)
        else:
            ops.to_fixed_point(a, out=o)

    for _ in range(args.warmup):
        for c in calls:
            run(c)
    stream = torch.cuda.current_stream(dev)
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in calls] for _ in range(args.steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for s in range(args.steps):
        for i, c in enumerate(calls):
            ev[s][i][0].record(stream)
            run(c)
            ev[s][i][1].record(stream)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps
    step_bytes = w_bytes + x_bytes
    q_ms = sum(ev[s][0][0].elapsed_time(ev[s][0][1]) for s in range(args.steps)) / args.steps
    f_ms = sum(ev[s][1][0].elapsed_time(ev[s][1][1]) for s in range(args.steps)) / args.steps
    q_launches = (len(layers) + 63) // 64
    kernels = {"quantize_kernel<Q>": (q_ms, w_bytes, q_launches),
               "to_fixed_kernel": (f_ms, x_bytes, 1)}
    name, (k_ms, k_bytes, k_launches) = max(kernels.items(), key=lambda kv: kv[1][0])
    achieved = k_bytes / (k_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                "kernel": name, "launches_per_step": k_launches,
                "avg_launch_ms": round(k_ms / k_launches, 5),
                "algorithmic_bytes_per_launch": k_bytes // k_launches,
                "per_kernel_gbs": {k: round(b / (m * 1e-3) / 1e9, 1) for k, (m, b, _) in kernels.items()},
                "timed_span": "library call per launch (one kernel each)"}
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        wn = [W.gen_float_weights(L.k, L.crs, seed=1000 + i) for i, L in enumerate(layers)]
        xn = W.gen_float_acts(nx, seed=5)
        t = time.perf_counter()
        passes = 0
        while True:
            for w in wn:
                oracle.pack_codes(oracle.quantize_q(w))
            oracle.to_fixed(xn)
            passes += 1
            if time.perf_counter() - t > args.cpu_seconds / 2:
                break
        dt = time.perf_counter() - t
        cpu = {"value": round(passes * step_bytes / dt / 1e9, 3), "unit": "GB/s", "cores": 1,
               "kind": "oracle", "sample": f"{passes} whole step(s) ({dt:.1f} s)"}
    out = {
        "metric": "GB/s of float-to-code conversion (weights) and fixed-point rounding (input)",
        "value": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32->u5/i32",
        "data": "synthetic",
        "config": {"workload": "resnet50_weights_and_input_n128", "weight_tensors": len(layers),
                   "weights": sum(L.k * L.crs for L in layers), "input_elements": nx,
                   "bytes_per_step": step_bytes, "parallelism": "single GPU"},
        "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def bench_network(args):
    """One step = one forward pass of the network over the batch (every op on the GPU,
    input resident in HBM); reported in images/s, with the shift convolutions'
    rate against the VALU roofline."""
    import torch
    from paper_1905_13298_amd import workloads as W
    from paper_1905_13298_amd.network import ShiftNetwork

    n = NETWORK_WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    graph, params = W.resnet18_graph(n), W.resnet18_params(n)
    x = torch.from_numpy(W.gen_images(n)).to(dev)
    stream = torch.cuda.current_stream(dev)
    conv_idx = [i for i, op in enumerate(graph) if op["op"] in ("conv", "linear")]
    sac = sum(graph[i]["layer"].sac for i in conv_idx)
    nz = sum(graph[i]["layer"].sac * float(np.mean((params[graph[i]["layer"].name]["codes"] & 15) != 15))
             for i in conv_idx)

    step_calls = {}

    def timed(net, name):
        calls = []
        buf = {"x": x}
        for op in graph:
            calls.append(lambda op=op: net.run_op(op, buf))
        step_calls[name] = (calls, buf)
        return time_layers(calls, args.steps, args.warmup, stream)

    nets = {"runtime": ShiftNetwork(graph, params, device=dev)}
    if args.path == "jit":
        nets["jit"] = ShiftNetwork(graph, params, device=dev, jit=True)
        a_out = nets["runtime"].forward(x, keep=True)
        b_out = nets["jit"].forward(x, keep=True)
        for op in graph:
            if not torch.equal(a_out[op["dst"]], b_out[op["dst"]]):
                raise SystemExit(f"{op['dst']}: weight-specialised and runtime outputs differ")
        del a_out, b_out
    results = {p: timed(net, p) for p, net in nets.items()}
    ms_per_step, d = results[args.path]
    timing = {"mode": "eager", "eager_ms_per_step": round(ms_per_step, 5)}
    if args.path == "jit" and not args.eager:
        # every op writes a buffer of its own that the network keeps: the graph's
        # outputs are those buffers
        calls, buf = step_calls["jit"]
        ms_per_step, rep = time_graph(calls, [buf[op["dst"]] for op in graph], args.steps, args.warmup)
        timing = {"mode": "HIP graph of consecutive steps, replayed", "steps_per_graph": rep,
                  "graph_ms_per_step": round(ms_per_step, 5), "eager_ms_per_step": timing["eager_ms_per_step"]}
    op_ms = d.mean(axis=0)
    conv_ms = float(sum(op_ms[i] for i in conv_idx))
    per_kind = {}
    for i, op in enumerate(graph):
        per_kind[op["op"]] = round(per_kind.get(op["op"], 0.0) + float(op_ms[i]), 4)
    common = {"traffic": None, "launches_per_step": len(conv_idx),
              "avg_launch_ms": round(conv_ms / len(conv_idx), 5), "sac_per_launch_avg": sac // len(conv_idx),
              "dense_tsac_s": round(sac / (conv_ms * 1e-3) / 1e12, 4)}
    if args.path == "jit":
        achieved = nz / (conv_ms * 1e-3) / 1e12
        roofline = {"bound": "alu", "achieved": round(achieved, 4), "peak": round(VOP2_OPS_PEAK_T, 4),
                    "unit": "T int32 ops/s", "frac": round(achieved / VOP2_OPS_PEAK_T, 4), **common,
                    "work_unit": "one int32 VOP2 add/sub per non-zero weight term",
                    "entry_points": list(JIT_ENTRY_POINTS),
                    "kernel": "weight-specialised convolutions with fused epilogue",
                    "timed_span": "library call per layer"}
    else:
        achieved = sac / (conv_ms * 1e-3) / 1e12
        roofline = {"bound": "alu", "achieved": round(achieved, 4), "peak": SAC_PEAK_T,
                    "unit": "TSAC/s", "frac": round(achieved / SAC_PEAK_T, 4), **common,
                    "work_unit": "dense shift-accumulate, 2 int32 VALU ops each",
                    "kernel": "shift convolutions with fused epilogue (all 21 layers)",
                    "timed_span": "library call per layer (weight decode + conv + fused epilogue)"}
    runtime = None
    if args.path == "jit":
        rt_ms = results["runtime"][0]
        runtime = {"ms_per_step": round(rt_ms, 4), "value": round(n / (rt_ms * 1e-3), 1),
                   "unit": "images/s"}
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        nc = 8
        xs = W.gen_images(nc)
        pc = W.resnet18_params(nc)
        gc = W.resnet18_graph(nc)
        t = time.perf_counter()
        oracle.network_forward(gc, pc, xs)
        dt = time.perf_counter() - t
        cpu = {"value": round(nc / dt, 3), "unit": "images/s", "cores": oracle.max_threads(),
               "kind": "oracle", "sample": f"one forward pass over {nc} images ({dt:.1f} s)"}
    ips = n / (ms_per_step * 1e-3)
    out = {
        "metric": "images/s of a ResNet-18 forward pass with shift convolutions (chained, fused epilogues)",
        "value": round(ips, 1), "unit": "images/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "ms_per_image": round(ms_per_step / n, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "i32",
        "data": "synthetic", "path": args.path,
        "config": {"workload": f"resnet18_forward_n{n}_224", "batch": n, "ops": len(graph),
                   "sac_per_step": sac, "nonzero_sac_per_step": int(nz), "frac_bits": W.FRAC_BITS,
                   "parallelism": "single GPU"},
        "timing": timing,
        "ms_by_op": per_kind, "roofline": roofline, "runtime_weights": runtime, "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def gen_grad(L, seed: int, index: int) -> np.ndarray:
    """Signed output gradient of a layer: rint(N(0, 1) * 2^16), int32 (F = 16)."""
    rng = np.random.default_rng([seed, index, 7])
    return np.rint(rng.standard_normal(L.y_shape, dtype=np.float32) * 65536.0).astype(np.int32)


def bench_backward(args):
    """One step = the input gradient of every layer (the stem aside) on its own
    seeded output gradient, all resident in HBM; dense shift-accumulates as for the
    forward pass (one term per forward connection). Path jit: a weight-specialised
    plan per layer (made at setup, stride phases as generated kernels) where one is
    preferred; path runtime: ds_conv2d_shift_backward_data / ds_linear_shift_backward_data."""
    import torch
    from paper_1905_13298_amd import ops
    from paper_1905_13298_amd import workloads as W

    cfg = BACKWARD_WORKLOADS[args.workload]
    seed = W.CONFIG_SEEDS[cfg]
    layers = [(li, L) for li, L in enumerate(W.config_layers(cfg)) if L.name != "conv1"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    rt_calls, calls, plans, names, nonzero, keep = [], [], [], [], [], []
    for li, L in layers:
        codes = W.gen_codes(L, seed, li)
        nonzero.append(float(np.mean((codes & 15) != 15)))
        wph = ops.pack_shift_weights(codes)
        wp = torch.from_numpy(wph.view(np.int32)).to(dev)
        dy = torch.from_numpy(gen_grad(L, seed, li)).to(dev)
        dx = torch.empty(L.x_shape, dtype=torch.int32, device=dev)
        if L.kind == "linear":
            rt = lambda dy=dy, wp=wp, dx=dx, L=L: ops.linear_shift_backward_data(dy, wp, L.c, out=dx)
            names.append(ops.describe_conv2d_backward_data(L.n, L.c, 1, 1, L.k, 1))
            fx, kern, st_, pd_, dy4 = (L.n, L.c, 1, 1), 1, 1, 0, dy.view(L.n, L.k, 1, 1)
        else:
            rt = lambda dy=dy, wp=wp, dx=dx, L=L: ops.conv2d_shift_backward_data(
                dy, wp, L.x_shape, (L.r, L.s), L.stride, L.pad, out=dx)
            names.append(ops.describe_conv2d_backward_data(*L.x_shape, L.k, (L.r, L.s), L.stride, L.pad))
            fx, kern, st_, pd_, dy4 = L.x_shape, (L.r, L.s), L.stride, L.pad, dy
        rt_calls.append(rt)
        plan = None
        if args.path == "jit":
            try:
                plan = ops.JitConvBackwardData(wph, fx, kern, st_, pd_)
            except ops.DeepShiftError:
                plan = None
            if plan is not None and not plan.preferred:
                plan.close()
                plan = None
        plans.append(plan)
        if plan is None:
            calls.append(rt)
        else:
            calls.append(lambda plan=plan, dy4=dy4, dx=dx: plan(dy4, out=dx.view(plan.y_shape)))
        keep.append((dy, wp, dx))
    torch.cuda.synchronize()
    if args.path == "jit":
        for i, (c_, r_) in enumerate(zip(calls, rt_calls)):
            c_()
            a_ = keep[i][2].clone()
            r_()
            if not torch.equal(a_, keep[i][2]):
                raise SystemExit(f"{layers[i][1].name}: plan and runtime input gradients differ")
        torch.cuda.synchronize()
    ms_per_step, d = time_layers(calls, args.steps, args.warmup, stream)
    timing = {"mode": "eager", "eager_ms_per_step": round(ms_per_step, 5)}
    if args.path == "jit" and not args.eager and all(p is not None for p in plans):
        ms_per_step, rep = time_graph(calls, [k[2] for k in keep], args.steps, args.warmup)
        timing = {"mode": "HIP graph of consecutive steps, replayed", "steps_per_graph": rep,
                  "graph_ms_per_step": round(ms_per_step, 5), "eager_ms_per_step": timing["eager_ms_per_step"]}
    sac_step = sum(L.sac for _, L in layers)
    nz_step = sum(L.sac * f for (_, L), f in zip(layers, nonzero))
    value = sac_step / (ms_per_step * 1e-3) / 1e9
    groups = {}
    for i, (li, L) in enumerate(layers):
        gname = JIT_KERNEL if plans[i] is not None else names[i]
        g = groups.setdefault(gname, {"sac": 0, "nz": 0.0, "ms": 0.0, "launches": 0, "bytes": 0})
        g["sac"] += L.sac
        g["nz"] += L.sac * nonzero[i]
        g["ms"] += float(d[:, i].mean())
        g["launches"] += 1
        g["bytes"] += algorithmic_bytes(L)
    name, g = max(groups.items(), key=lambda kv: kv[1]["ms"])
    common = {"traffic": None, "kernel": name, "launches_per_step": g["launches"],
              "avg_launch_ms": round(g["ms"] / g["launches"], 5),
              "sac_per_launch_avg": g["sac"] // g["launches"],
              "algorithmic_bytes_per_launch": g["bytes"] // g["launches"]}
    if name == JIT_KERNEL:
        nz = g["nz"] / (g["ms"] * 1e-3) / 1e12
        roofline = {"bound": "alu", "achieved": round(nz, 4), "peak": round(VOP2_OPS_PEAK_T, 4),
                    "unit": "T int32 ops/s", "frac": round(nz / VOP2_OPS_PEAK_T, 4), **common,
                    "work_unit": "one int32 VOP2 add/sub per non-zero weight term",
                    "entry_points": list(JIT_ENTRY_POINTS),
                    "dense_tsac_s": round(g["sac"] / (g["ms"] * 1e-3) / 1e12, 4),
                    "timed_span": "library call per layer (zero fills, the phases' generated kernels)"}
    else:
        achieved = g["sac"] / (g["ms"] * 1e-3) / 1e12
        roofline = {"bound": "alu", "achieved": round(achieved, 4), "peak": round(SAC_PEAK_T, 4),
                    "unit": "TSAC/s", "frac": round(achieved / SAC_PEAK_T, 4), **common,
                    "work_unit": "dense shift-accumulate, 2 int32 VALU ops each (3 on chunks holding a negative value)",
                    "timed_span": "library call per layer (code re-pack, weight decode, fill, phase kernels)"}
    runtime = None
    if args.path == "jit" and not args.no_runtime:
        rt_ms, _ = time_layers(rt_calls, args.steps, args.warmup, stream)
        runtime = {"ms_per_step": round(rt_ms, 4), "value": round(sac_step / (rt_ms * 1e-3) / 1e9, 2),
                   "unit": "GSAC/s"}
    per_layer = [{"layer": L.name, "plan": names[i], "jit": plans[i] is not None, "sac": L.sac,
                  "ms_median": float(np.median(d[:, i])),
                  "gsac_s": L.sac / (float(np.median(d[:, i])) * 1e-3) / 1e9}
                 for i, (li, L) in enumerate(layers)]
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        del calls, rt_calls, keep
        for p in plans:
            if p is not None:
                p.close()
        torch.cuda.empty_cache()
        nb = 2
        t_total, s_total, passes = 0.0, 0, 0
        while True:
            for li, L in layers:
                Ls = L.with_batch(min(nb, L.n))
                codes = W.gen_codes(L, seed, li)
                dy = gen_grad(Ls, seed, li)
                t = time.perf_counter()
                if L.kind == "linear":
                    oracle.linear_shift_backward_data(dy, codes)
                else:
                    oracle.conv2d_shift_backward_data(dy, codes, Ls.x_shape, r=L.r, s=L.s,
                                                      stride=L.stride, pad=L.pad)
                t_total += time.perf_counter() - t
                s_total += Ls.sac
            passes += 1
            if t_total >= args.cpu_seconds:
                break
        cpu = {"value": round(s_total / t_total / 1e9, 3), "unit": "GSAC/s", "cores": oracle.max_threads(),
               "kind": "oracle", "sample": f"{passes} pass(es) over the layers at batch {nb} "
                                           f"({s_total / 1e9:.2f} G SAC, {t_total:.1f} s)"}
    out = {
        "metric": "G shift-accumulates/s of the input gradient (backward data) per layer on one MI355X",
        "value": round(value, 2), "unit": "GSAC/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "i32", "data": "synthetic",
        **({"frac_vop2_peak_nonzero": round(nz_step / (ms_per_step * 1e-3) / 1e12 / VOP2_OPS_PEAK_T, 4)}
           if args.path == "jit" else {"frac_sac_peak": round(value / 1000.0 / SAC_PEAK_T, 4)}),
        "path": args.path,
        "config": {"workload": W.CONFIG_NAMES[cfg] + "_backward_data", "layers": len(layers),
                   "batch": layers[0][1].n, "frac_bits": W.FRAC_BITS, "sac_per_step": sac_step,
                   "grad": "rint(N(0,1) * 2^16), signed", "parallelism": "single GPU"},
        "timing": timing,
        "roofline": roofline, "runtime_weights": runtime, "cpu_baseline": cpu,
    }
    if args.layers_out:
        with open(args.layers_out, "w") as f:
            json.dump({"workload": args.workload, "layers": per_layer}, f, indent=1)
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.copy_only:
        copy_only(args.copy_only)
        return
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, args.pmc_copy_bytes, args.workload, args.path, args.pmc_out)
        return
    if args.sq_summary:
        sq_summary(args.sq_summary, args.workload, args.path)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the shift operators need "
              "no cross-GPU exchange for a layer, see the design notes for how they shard.",
              file=sys.stderr)
        sys.exit(2)

    if args.steps is None and args.workload not in WORKLOADS and args.workload not in PROBE_WORKLOADS \
            and args.workload not in MODEL_WORKLOADS:
        args.steps = 24
    if args.workload in CONVERT_WORKLOADS:
        bench_convert(args)
        return
    if args.workload in NETWORK_WORKLOADS:
        bench_network(args)
        return
    if args.workload in BACKWARD_WORKLOADS:
        bench_backward(args)
        return

    bench_layers(args)


def jit_supported(L) -> bool:
    """Layers a weight-specialised plan covers: every ConvShift (windows over 3 x 3
    through a zero-padded copy of x) and LinearShift."""
    return L.kind in ("conv", "linear")


def group_name(L, path: str, planned: bool | None = None) -> str:
    """The kernel a layer's call is accounted to (one kernel instance). `planned`:
    whether the layer runs a weight-specialised plan (default: whenever one covers it)."""
    if path == "jit" and (jit_supported(L) if planned is None else planned):
        return JIT_KERNEL
    return kernel_variant(L).rsplit(" splits", 1)[0]


def time_graph(calls, outs, steps, warmup):
    """The step (every call in order) captured in a HIP graph and replayed.
    Launching a step from the host costs microseconds per call, which for the
    shortest layers is more than their kernels; a graph launches the same
    kernels (plans use no memset and allocate nothing when run). A graph launch
    itself costs tens of microseconds, so a graph holds R consecutive steps, R
    the largest divisor of `steps` that keeps it within 64 calls: `warmup`
    untimed steps, then steps / R replays between two HIP events. The outputs
    of the first and the last replay must equal those of the eager calls.
    Returns (ms per step, R)."""
    import torch
    per = max(1, 64 // max(1, len(calls)))
    rep = max(r for r in range(1, min(per, steps) + 1) if steps % r == 0)
    for c in calls:
        c()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            for _ in range(rep):
                for c in calls:
                    c()
    torch.cuda.synchronize()

    def check(when):
        for o, r in zip(outs, ref):
            if not torch.equal(o, r):
                raise SystemExit(f"graph replay ({when}) differs from the eager calls")
    for o in outs:
        o.fill_(-1)
    g.replay()
    torch.cuda.synchronize()
    check("first")
    for _ in range(-(-warmup // rep)):
        g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for _ in range(steps // rep):
        g.replay()
    t_end.record(stream)
    torch.cuda.synchronize()
    check("last")
    del g
    return t_start.elapsed_time(t_end) / steps, rep


def time_layers(calls, steps, warmup, stream):
    """Run every call `warmup` times untimed, then `steps` timed passes between
    two HIP events on `stream` (the step time), then `steps` more passes with
    HIP events around each call (the per-call durations, which the events
    themselves lengthen a little: a chained ResNet-18 step of 1.44 ms took 1.66 ms
    with an event pair around each of its 30 ops). Returns (ms per step, per-call
    durations [steps][calls] in ms)."""
    import torch
    for _ in range(warmup):
        for c in calls:
            c()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for _ in range(steps):
        for c in calls:
            c()
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_end) / steps
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in calls] for _ in range(steps)]
    for s in range(steps):
        for i, c in enumerate(calls):
            ev[s][i][0].record(stream)
            c()
            ev[s][i][1].record(stream)
    torch.cuda.synchronize()
    d = np.array([[a.elapsed_time(b) for a, b in row] for row in ev])
    return ms_per_step, d


def roofline_of(layers, d, path, nonzero, planned=None, act_bits=32, workload=None):
    """Roofline record of the kernel with the most time per step, from the
    per-call durations `d` [steps][layers]; planned[i]: layer i runs a plan."""
    groups = {}
    for li, L in enumerate(layers):
        g = groups.setdefault(group_name(L, path, None if planned is None else planned[li]), {"sac": 0, "nz": 0.0, "ms": 0.0, "launches": 0,
                                                    "bytes": 0})
        g["sac"] += L.sac
        g["nz"] += L.sac * nonzero[li]
        g["ms"] += float(d[:, li].mean())
        g["launches"] += 1
        g["bytes"] += algorithmic_bytes(L, act_bits)
    name, g = max(groups.items(), key=lambda kv: kv[1]["ms"])
    traffic = measured_traffic(name, "jit" if name == JIT_KERNEL else "runtime", workload) \
        if act_bits == 32 and workload else None
    common = {
        "traffic": None if traffic is None else int(traffic),
        "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
        "algorithmic_bytes_per_launch": g["bytes"] // g["launches"],
        "kernel": name, "launches_per_step": g["launches"],
        "avg_launch_ms": round(g["ms"] / g["launches"], 5),
        "sac_per_launch_avg": g["sac"] // g["launches"],
        "hbm_gbs_algorithmic": round(g["bytes"] / (g["ms"] * 1e-3) / 1e9, 1),
    }
    dense = g["sac"] / (g["ms"] * 1e-3) / 1e12
    if name == JIT_KERNEL:
        # Weight-specialised code: one VOP2 add or subtract per non-zero weight term
        # is the floor (the shifts are shared by 64 output channels, zero weights cost
        # nothing), so the roofline counts non-zero terms against the VOP2 lane-op peak.
        nz = g["nz"] / (g["ms"] * 1e-3) / 1e12
        return {"bound": "alu", "achieved": round(nz, 4), "peak": round(VOP2_OPS_PEAK_T, 4),
                "unit": "T int32 ops/s", "frac": round(nz / VOP2_OPS_PEAK_T, 4),
                "frac_of_64_lanes_per_cu_clk": round(nz / INT32_OPS_PEAK_T, 4), **common,
                "work_unit": "one int32 VOP2 add/sub per non-zero weight term",
                "entry_points": list(JIT_ENTRY_POINTS),
                "nonzero_sac_per_launch_avg": int(g["nz"] // g["launches"]),
                "dense_tsac_s": round(dense, 4),
                "timed_span": "library call per launch (split-K fill pass, or for a LinearShift on x^T the transposing passes, + generated kernel)"}
    return {"bound": "alu", "achieved": round(dense, 4), "peak": round(SAC_PEAK_T, 4),
            "unit": "TSAC/s", "frac": round(dense / SAC_PEAK_T, 4), **common,
            "work_unit": "dense shift-accumulate, 2 int32 VALU ops each",
            "int32_ops_frac": round(2 * dense / INT32_OPS_PEAK_T, 4),
            "timed_span": "library call (weight decode + main kernel) per launch"}


def bench_layers(args):
    import torch
    from paper_1905_13298_amd import ops
    from paper_1905_13298_amd import workloads as W

    if args.workload in PROBE_WORKLOADS:
        cfg, seed, layers = None, 99, [W.VALU_PROBE]
    elif args.workload in MODEL_WORKLOADS:
        cfg, seed, layers = None, 98, [W.LINEAR_25088_B1]
    else:
        cfg = WORKLOADS[args.workload]
        seed = W.CONFIG_SEEDS[cfg]
        layers = W.config_layers(cfg)
    if args.steps is None:
        # A single layer's step lasts microseconds and a graph launch tens of
        # them: 640 steps (10 graphs of 64) keep launches a small part of the
        # timed region. A network's step lasts milliseconds: 24 steps, in graphs
        # of up to 64 calls (3 steps of ResNet-18, which read 5-8 % faster per
        # step than graphs of one step on MI355X).
        args.steps = 640 if len(layers) == 1 else 24
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    # ---- inputs resident in HBM before timing; weight-specialised plans are made
    # here too (host code generation, once per layer, like packing the weights)
    t0 = time.time()
    res, plans, nonzero, model, rejected = [], [], [], [], []
    plan_s = 0.0
    act = args.act_bits
    if act != 32 and args.path != "jit":
        raise SystemExit("--act-bits 16/8 runs on weight-specialised plans (--path jit)")
    for li, L in enumerate(layers):
        x, codes, bias = W.gen_layer(L, seed, li, act_bits=act)
        nonzero.append(float(np.mean((codes & 15) != 15)))
        wp = ops.pack_shift_weights(codes)
        xt = torch.from_numpy(x).to(dev)
        wt = torch.from_numpy(wp.view(np.int32)).to(dev)
        bt = None if bias is None else torch.from_numpy(bias).to(dev)
        yt = torch.empty(L.y_shape, dtype=torch.int32, device=dev)
        res.append((L, xt, wt, bt, yt))
        plan = None
        if args.path == "jit" and jit_supported(L):
            tp = time.time()
            plan = ops.layer_plan(L, wp, bias, act_bits=act)
            plan_s += time.time() - tp
            model.append((plan.estimate_us(), plan.runtime_estimate_us(), plan.preferred,
                          {"code_bytes": plan.code_bytes, "segments": plan.segments, "splits": plan.splits,
                           "channels": plan.channels, "wsplit": plan.wsplit, "pixel_groups": plan.pixel_groups,
                           "pixel_tiles": plan.pixel_tiles, "transposed": plan.transposed}))
            if not plan.preferred:
                if args.time_rejected:
                    rejected.append((len(plans), plan))
                else:
                    plan.close()
                plan = None
        else:
            model.append(None)
        plans.append(plan)
        del x, codes, bias
    torch.cuda.synchronize()
    print(f"# inputs ready in {time.time() - t0:.1f} s (plans {plan_s:.1f} s)", file=sys.stderr, flush=True)

    def runtime_call(L, xt, wt, bt, yt):
        # The runtime kernel reads int32: narrow activations are widened (sign-extended)
        # for it, which is their value -- it then checks the plans' outputs.
        x32 = xt if xt.dtype == torch.int32 else xt.to(torch.int32)
        if L.kind == "linear":
            return lambda: ops.linear_shift(x32, wt, bt, out=yt)
        return lambda: ops.conv2d_shift(x32, wt, bt, (L.r, L.s), L.stride, L.pad, out=yt)

    def jit_call(plan, L, xt, wt, bt, yt):
        if plan is None:
            return runtime_call(L, xt, wt, bt, yt)
        return lambda: ops.run_layer_plan(plan, L, xt, out=yt)

    runtime_calls = [runtime_call(*r) for r in res]
    sac_step = sum(L.sac for L in layers)
    nz_step = sum(L.sac * f for L, f in zip(layers, nonzero))

    if args.path == "jit":
        jit_calls = [jit_call(p, *r) for p, r in zip(plans, res)]
        # Both paths must agree on every output before either is timed.
        for c in jit_calls:
            c()
        jit_out = [r[4].clone() for r in res]
        for c in runtime_calls:
            c()
        torch.cuda.synchronize()
        for (L, *_r, yt), yj in zip(res, jit_out):
            if not torch.equal(yt, yj):
                raise SystemExit(f"{L.name}: weight-specialised and runtime outputs differ")
        del jit_out
        ms_per_step, d = time_layers(jit_calls, args.steps, args.warmup, stream)
    else:
        ms_per_step, d = time_layers(runtime_calls, args.steps, args.warmup, stream)
    timing = {"mode": "eager", "eager_ms_per_step": round(ms_per_step, 5)}
    # Graph replay when every call launches kernels only: plans, and LinearShift
    # layers on the small-batch runtime kernel (no scratch; its fill pass is a kernel).
    def graphable(L, plan):
        return plan is not None or (L.kind == "linear" and ops.describe_conv2d(L.n, L.c, 1, 1, L.k, 1) == "rows")
    if args.path == "jit" and not args.eager and all(graphable(L, p) for L, p in zip(layers, plans)):
        ms_per_step, rep = time_graph(jit_calls, [r[4] for r in res], args.steps, args.warmup)
        timing = {"mode": "HIP graph of consecutive steps, replayed", "steps_per_graph": rep,
                  "graph_ms_per_step": round(ms_per_step, 5), "eager_ms_per_step": timing["eager_ms_per_step"]}
    value = sac_step / (ms_per_step * 1e-3) / 1e9
    planned = [p is not None for p in plans]
    wl_name = W.CONFIG_NAMES[cfg] if cfg is not None else args.workload
    roofline = roofline_of(layers, d, args.path, nonzero, planned, act, workload=wl_name)

    runtime = None
    d_rt = d
    if args.path == "jit" and not args.no_runtime and act == 32:
        rt_ms, d_rt = time_layers(runtime_calls, args.steps, args.warmup, stream)
        rt_value = sac_step / (rt_ms * 1e-3) / 1e9
        runtime = {"ms_per_step": round(rt_ms, 4), "value": round(rt_value, 2), "unit": "GSAC/s",
                   "frac_sac_peak": round(rt_value / 1000.0 / SAC_PEAK_T, 4),
                   "roofline": roofline_of(layers, d_rt, "runtime", nonzero, workload=wl_name)}

    per_layer = []
    fr = [L.sac * nonzero[li] / (float(np.median(d[:, li])) * 1e-3) / 1e12 / VOP2_OPS_PEAK_T
          for li, L in enumerate(layers)]
    order = np.argsort(fr)
    layer_summary = {
        "layers": len(layers),
        "frac_basis": ("non-zero terms / (median call time x 78.64 T VOP2 lane-ops/s)" if args.path == "jit"
                       else "dense SAC / (median call time x 19.66 T SAC/s)"),
        "min_frac": round(float(min(fr)), 4) if args.path == "jit" else None,
        "median_frac": round(float(np.median(fr)), 4) if args.path == "jit" else None,
        "layers_frac_ge_0_6": int(sum(f >= 0.6 for f in fr)) if args.path == "jit" else None,
        "worst": [[layers[i].name, round(float(fr[i]), 3)] for i in order[:5]] if args.path == "jit" else None,
        "nonzero_tsac_s": round(nz_step / (ms_per_step * 1e-3) / 1e12, 3),
        "per_layer": [[L.name, round(float(np.median(d[:, li])), 5),
                       round(L.sac / (float(np.median(d[:, li])) * 1e-3) / 1e9, 1)]
                      for li, L in enumerate(layers)],
        "per_layer_fields": ["layer", "median ms", "dense G SAC/s"],
    }
    if args.path != "jit":
        frs = [L.sac / (float(np.median(d[:, li])) * 1e-3) / 1e12 / SAC_PEAK_T for li, L in enumerate(layers)]
        layer_summary.update({"min_frac": round(float(min(frs)), 4), "median_frac": round(float(np.median(frs)), 4),
                              "layers_frac_ge_0_6": int(sum(f >= 0.6 for f in frs)),
                              "worst": [[layers[i].name, round(float(frs[i]), 3)] for i in np.argsort(frs)[:5]]})
    for li, L in enumerate(layers):
        med = float(np.median(d[:, li]))
        row = {
            "layer": L.name, "kind": L.kind, "kernel": group_name(L, args.path, planned[li]),
            "variant": kernel_variant(L),
            "shape": {"n": L.n, "c": L.c, "h": L.h, "w": L.w, "k": L.k, "r": L.r, "s": L.s,
                      "stride": L.stride, "pad": L.pad},
            "sac": L.sac, "nonzero_frac": round(nonzero[li], 4), "ms_median": med,
            "ms_mean": float(d[:, li].mean()), "ms_min": float(d[:, li].min()),
            "gsac_s": L.sac / (med * 1e-3) / 1e9,
            "frac_sac_peak": L.sac / (med * 1e-3) / 1e12 / SAC_PEAK_T,
            "frac_vop2_peak_nonzero": L.sac * nonzero[li] / (med * 1e-3) / 1e12 / VOP2_OPS_PEAK_T,
            "hbm_gbs": algorithmic_bytes(L, act) / (med * 1e-3) / 1e9,
        }
        if runtime is not None:
            row["runtime_ms_median"] = float(np.median(d_rt[:, li]))
        if model[li] is not None:
            row["plan_model_us"] = round(model[li][0], 2)
            row["runtime_model_us"] = round(model[li][1], 2)
            row["plan_preferred"] = model[li][2]
            row["plan_layout"] = model[li][3]
        per_layer.append(row)
    # Plans the cost model rejected, timed on their own (each checked first).
    for li, plan in rejected:
        L, xt, wt, bt, yt = res[li]
        ref = yt.clone()
        runtime_call(L, xt, wt, bt, yt)()
        ref.copy_(yt)
        ops.run_layer_plan(plan, L, xt, out=yt)
        torch.cuda.synchronize()
        if not torch.equal(yt, ref):
            raise SystemExit(f"{L.name}: rejected plan and runtime outputs differ")
        _, d_rej = time_layers([lambda plan=plan, L=L, xt=xt, yt=yt: ops.run_layer_plan(plan, L, xt, out=yt)],
                               args.steps, args.warmup, stream)
        per_layer[li]["rejected_plan_ms_median"] = float(np.median(d_rej[:, 0]))
        plan.close()

    # ---- multiplication-based comparison, each against the shift path of the same tiling
    mul = None
    if not args.no_mul and act == 32:
        rt_shift_ms = runtime["ms_per_step"] if runtime is not None else (
            ms_per_step if args.path == "runtime" else time_layers(runtime_calls, args.steps, 1, stream)[0])
        # (both sides of each comparison timed as eager calls)
        mul = mul_comparison(args, res, layers, seed, stream, rt_shift_ms,
                             timing["eager_ms_per_step"] if args.path == "jit" else None)

    # ---- CPU baseline: the oracle on the host cores, same layers at a small batch
    cpu = None
    if not args.no_cpu_baseline:
        del res, plans, runtime_calls
        if args.path == "jit":
            del jit_calls
        torch.cuda.empty_cache()
        cpu = cpu_baseline(args, cfg, seed, layers, act) if cfg is not None else None

    path_desc = ("weight-specialised plans (code generated per layer at setup), the runtime "
                 "kernel where a plan is not preferred"
                 if args.path == "jit" else "runtime weights (ds_conv2d_shift / ds_linear_shift)")
    out = {
        "metric": "G shift-accumulates/s per layer and % of int32 VALU peak on one MI355X",
        "value": round(value, 2), "unit": "GSAC/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "i32" if act == 32 else f"i{act}->i32",
        "data": "synthetic",
        **({"frac_vop2_peak_nonzero": round(nz_step / (ms_per_step * 1e-3) / 1e12 / VOP2_OPS_PEAK_T, 4)}
           if args.path == "jit" else {"frac_sac_peak": round(value / 1000.0 / SAC_PEAK_T, 4)}),
        "path": path_desc,
        "config": {"workload": (W.CONFIG_NAMES[cfg] if cfg is not None else args.workload)
                   + ("" if act == 32 else f"_act{act}"),
                   "layers": len(layers), "batch": layers[0].n, "frac_bits": W.ACT_FRAC_BITS[act],
                   "act_bits": act,
                   "sac_per_step": sac_step, "nonzero_sac_per_step": int(nz_step),
                   "parallelism": "single GPU"},
        "timing": timing,
        "roofline": roofline, "layer_summary": layer_summary, "runtime_weights": runtime,
        "cpu_baseline": cpu, "mul_comparison": mul,
    }
    if args.layers_out:
        with open(args.layers_out, "w") as f:
            json.dump({"workload": W.CONFIG_NAMES[cfg] if cfg is not None else args.workload,
                       "path": args.path, "layers": per_layer}, f, indent=1)
    print(json.dumps(out), flush=True)


def mul_comparison(args, res, layers, seed, stream, rt_shift_ms, plan_shift_ms):
    """The multiplication-based comparison (the paper's Section 6 times its shift
    kernels against a multiplication kernel), each timed against the shift path
    of the same tiling: the runtime kernel's tiling with an int32 multiply-add
    (v_mul_lo_u32 + v_add3_u32, 1.5 instructions per term) and with a 24-bit one
    (v_mad_i32_i24), on random 16-bit weights; and the plans' tiling, with each
    layer's own weights as 14-bit fixed-point integers sign * 2^(14 - shift)
    baked into the code, one v_mad_i32_i24 per non-zero weight."""
    import torch
    from paper_1905_13298_amd import ops
    from paper_1905_13298_amd import workloads as W
    dev = res[0][1].device
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    i32_calls, i24_calls = [], []
    for (L, xt, wt, bt, yt) in res:
        wm = torch.randint(-(1 << 15), 1 << 15, (L.k, L.crs), dtype=torch.int32, device=dev, generator=g)
        for calls, m24 in ((i32_calls, False), (i24_calls, True)):
            if L.kind == "linear":
                calls.append(lambda xt=xt, wm=wm, bt=bt, yt=yt, m24=m24:
                             ops.linear_mul_i32(xt, wm, bt, out=yt, mul24=m24))
            else:
                calls.append(lambda L=L, xt=xt, wm=wm, bt=bt, yt=yt, m24=m24:
                             ops.conv2d_mul_i32(xt, wm, bt, (L.r, L.s), L.stride, L.pad, out=yt, mul24=m24))
    i32_ms, _ = time_layers(i32_calls, args.steps, 1, stream)
    i24_ms, _ = time_layers(i24_calls, args.steps, 1, stream)
    del i32_calls, i24_calls
    out = {"runtime_tiling": {
        "shift_ms": round(rt_shift_ms, 4), "mul_i32_ms": round(i32_ms, 4), "mul_i24_ms": round(i24_ms, 4),
        "shift_speedup_vs_mul_i32": round(i32_ms / rt_shift_ms, 3),
        "shift_speedup_vs_mul_i24": round(i24_ms / rt_shift_ms, 3),
        "inner_ops": {"shift": "v_ashrrev_i32 + v_xad_u32 per dense term",
                      "mul_i32": "v_mul_lo_u32 + v_add3_u32 (1.5 per term)", "mul_i24": "v_mad_i32_i24"}}}
    if plan_shift_ms is not None:
        plans, calls, mul_bytes = [], [], 0
        for li, (L, xt, wt, bt, yt) in enumerate(res):
            codes = W.gen_codes(L, seed, li)
            sh = (codes & 15).astype(np.int64)
            wv = np.where(sh == 15, 0, np.left_shift(1, 14 - np.minimum(sh, 14)))
            wv = np.where((codes >> 4) & 1, -wv, wv).astype(np.int32)
            bias = None if bt is None else bt.cpu().numpy()
            if L.kind == "linear":
                p = ops.JitConvMul(wv, (L.n, L.c, 1, 1), 1, 1, 0, bias=bias, device=dev)
                x4, y4 = xt.view(L.n, L.c, 1, 1), yt.view(L.n, L.k, 1, 1)
                calls.append(lambda p=p, x4=x4, y4=y4: p(x4, out=y4))
            else:
                p = ops.JitConvMul(wv, L.x_shape, (L.r, L.s), L.stride, L.pad, bias=bias, device=dev)
                calls.append(lambda p=p, xt=xt, yt=yt: p(xt, out=yt))
            mul_bytes += p.code_bytes
            plans.append(p)
        mp_ms, _ = time_layers(calls, args.steps, 1, stream)
        for p in plans:
            p.close()
        out["plan_tiling"] = {
            "shift_ms": round(plan_shift_ms, 4), "mul_i24_ms": round(mp_ms, 4),
            "shift_speedup": round(mp_ms / plan_shift_ms, 3), "mul_code_bytes": int(mul_bytes),
            "weights": "each layer's own weights as sign * 2^(14 - shift), zero weights skipped by both",
            "inner_ops": {"shift": "one v_add_u32/v_sub_u32 per non-zero term + shared v_ashrrev_i32",
                          "mul_i24": "one v_mad_i32_i24 per non-zero term (+ s_mov_b32 of the weight)"}}
    return out


def cpu_baseline(args, cfg, seed, layers, act_bits=32):
    """The oracle on the host's cores over whole passes of every layer at a small
    batch, for about args.cpu_seconds of oracle time."""
    import oracle
    from paper_1905_13298_amd import workloads as W
    nthreads = oracle.max_threads()
    cpu_batch = args.cpu_batch
    if cpu_batch is None:
        cpu_batch = {0: 8, 1: 1, 2: 256, 3: 8, 4: 8}[cfg]
    sample = [L.with_batch(min(cpu_batch, L.n)) for L in layers]
    cache_inputs = sum(4 * int(np.prod(L.x_shape)) for L in sample) < (2 << 30)
    cached = {}
    sample_sac = 0
    cpu_total = 0.0
    passes = 0
    wall0 = time.perf_counter()
    while True:
        for li, Ls in enumerate(sample):
            if li in cached:
                x, codes, bias = cached[li]
            else:
                x, codes, bias = W.gen_layer(Ls, seed, li, act_bits=act_bits)
                if cache_inputs:
                    cached[li] = (x, codes, bias)
            t1 = time.perf_counter()
            if Ls.kind == "linear":
                oracle.linear_shift(x, codes, bias)
            else:
                oracle.conv2d_shift(x, codes, bias, r=Ls.r, s=Ls.s, stride=Ls.stride, pad=Ls.pad)
            cpu_total += time.perf_counter() - t1
            sample_sac += Ls.sac
        passes += 1
        if cpu_total >= args.cpu_seconds or time.perf_counter() - wall0 > 3 * args.cpu_seconds:
            break
    cached.clear()
    return {"value": round(sample_sac / cpu_total / 1e9, 3), "unit": "GSAC/s",
            "cores": nthreads, "kind": "oracle",
            "sample": f"{passes} pass(es) over every layer of the workload at batch {cpu_batch} "
                      f"({sample_sac / 1e9:.2f} G SAC, {cpu_total:.1f} s)"}


if __name__ == "__main__":
    main()
