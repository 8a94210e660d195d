"""Chained inference: a network of shift convolutions run layer by layer on the GPU.

Interprets an op graph (see ``workloads.resnet18_graph``) with the library's
entry points: every convolution is one ``ds_conv2d_shift_fused`` call (shift
convolution, batch normalisation as a per-channel fixed-point affine map, the
residual add and ReLU in one kernel), pooling is ``ds_maxpool2d`` /
``ds_avgpool2d_global``, the classifier is ``ds_linear_shift``. Parameters are
uploaded once; activation buffers are allocated once per batch size and reused.

With ``jit=True`` the convolutions and the classifier run weight-specialised
plans (``ds_jit_conv_*``, made once here for the graph's batch size) with the
same fused epilogue where a plan is expected to be faster
(``JitConv.preferred``); ``jit="all"`` uses a plan for every layer. The results
are the same bit for bit. Calls at another batch size take the runtime kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import ops


class ShiftNetwork:
    def __init__(self, graph, params, device="cuda:0", mul_shift: int = 16, jit=False):
        self.graph = graph
        self.jit = jit
        self.dev = torch.device(device)
        self.mul_shift = mul_shift
        self.weights = {}
        self.plans = {}
        for op in graph:
            if op["op"] not in ("conv", "linear"):
                continue
            L = op["layer"]
            p = params[L.name]
            packed = torch.from_numpy(ops.pack_shift_weights(p["codes"]).view(np.int32)).to(self.dev)
            entry = {"w": packed}
            if op["op"] == "conv":
                mul, add = p["bn"]
                entry["mul"] = torch.from_numpy(np.ascontiguousarray(mul)).to(self.dev)
                entry["add"] = torch.from_numpy(np.ascontiguousarray(add)).to(self.dev)
            else:
                b = p.get("bias")
                entry["bias"] = None if b is None else torch.from_numpy(np.ascontiguousarray(b)).to(self.dev)
            self.weights[L.name] = entry
            if jit:
                self._make_plan(op, p)
        self._bufs = {}

    def _make_plan(self, op, p):
        L = op["layer"]
        wp = ops.pack_shift_weights(p["codes"])
        if op["op"] == "linear":
            plan = ops.JitConv(wp, (L.n, L.c, 1, 1), 1, 1, 0, bias=p.get("bias"), device=self.dev)
        else:
            mul, add = p["bn"]
            plan = ops.JitConv(wp, L.x_shape, (L.r, L.s), L.stride, L.pad, mul=mul, add=add,
                               mul_shift=self.mul_shift, residual=op["res"] is not None,
                               relu=op["relu"], device=self.dev)
        if plan.preferred or self.jit == "all":
            self.plans[L.name] = plan
        else:
            plan.close()

    def _out(self, name, shape):
        t = self._bufs.get(name)
        if t is None or tuple(t.shape) != tuple(shape):
            t = torch.empty(shape, dtype=torch.int32, device=self.dev)
            self._bufs[name] = t
        return t

    def run_op(self, op, buf):
        kind = op["op"]
        src = buf[op["src"]]
        if kind == "conv":
            L = op["layer"]
            w = self.weights[L.name]
            n, _, h, wd = src.shape
            oh, ow = ops.out_size(h, L.pad, L.r, L.stride), ops.out_size(wd, L.pad, L.s, L.stride)
            y = self._out(op["dst"], (n, L.k, oh, ow))
            res = buf[op["res"]] if op["res"] else None
            plan = self.plans.get(L.name)
            if plan is not None and tuple(src.shape) == plan.x_shape:
                plan(src, residual=res, out=y)
                buf[op["dst"]] = y
                return y
            ops.conv2d_shift_fused(src, w["w"], None, (L.r, L.s), L.stride, L.pad, mul=w["mul"],
                                   add=w["add"], mul_shift=self.mul_shift, residual=res,
                                   relu=op["relu"], out=y)
        elif kind == "maxpool":
            n, c, h, wd = src.shape
            oh, ow = ops.out_size(h, op["pad"], op["r"], op["stride"]), ops.out_size(wd, op["pad"], op["r"], op["stride"])
            y = self._out(op["dst"], (n, c, oh, ow))
            ops.maxpool2d(src, op["r"], op["stride"], op["pad"], out=y)
        elif kind == "avgpool":
            y = self._out(op["dst"], tuple(src.shape[:2]))
            ops.avgpool2d_global(src, out=y)
        elif kind == "linear":
            L = op["layer"]
            w = self.weights[L.name]
            y = self._out(op["dst"], (src.shape[0], L.k))
            plan = self.plans.get(L.name)
            if plan is not None and (src.shape[0], src.shape[1], 1, 1) == plan.x_shape:
                plan(src.view(plan.x_shape), out=y.view(plan.y_shape))
            else:
                ops.linear_shift(src, w["w"], w["bias"], out=y)
        else:
            raise ValueError(kind)
        buf[op["dst"]] = y
        return y

    def forward(self, x: torch.Tensor, keep: bool = False):
        """x: device int32 [n, c, h, w] in fixed point; returns the last op's output
        (or every buffer, by name, when keep)."""
        buf = {"x": x}
        y = None
        for op in self.graph:
            y = self.run_op(op, buf)
        return buf if keep else y
