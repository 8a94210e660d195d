"""Seeded synthetic inputs and layer shapes for the shift operators.

This module is shared by the oracle-side tests and the HIP-side callers. It
holds random-number generation and shape tables only: it performs none of the
shift operators' arithmetic.

Data formats produced here (they are the library's input formats):

* activations: int32 fixed point with F = 16 fractional bits, i.e. the integer
  ``round(u * 2**16)`` for a real value ``u`` (the paper's 16.16 rounding of
  inputs and bias, Implementation section). ``numpy.rint`` (half to even) does
  the rounding.
* weight codes: uint8, ``code = sign << 4 | shift_code``. ``shift_code`` in
  0..14 means the power of two ``2**-shift_code``; 15 means a zero weight
  (either sign bit). ``sign = 1`` means the negated power. This is the 5-bit
  budget of one sign bit plus a 4-bit shift with shifts between 0 and -14
  (Implementation section).
* bias: int32 with the same F as the activations.

The five workloads follow the benchmark configurations of this project:

0. LinearShift batch 8, 256 -> 128, signed activations in U[-4, 4).
1. Conv2dShift N=1, 128 -> 128 channels, 28 x 28, 3 x 3, stride 1, pad 1.
2. LinearShift batch 256, 4096 -> 4096, activations in U[0, 2).
3. Every Conv2dShift layer of ResNet-18 plus its 512 -> 1000 LinearShift, N=32.
4. Every Conv2dShift layer of ResNet-50 plus its 2048 -> 1000 LinearShift,
   N=128, 20 % zero codes.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

FRAC_BITS = 16
_CHUNK = 1 << 22  # elements per independently seeded activation chunk


@dataclasses.dataclass(frozen=True)
class Layer:
    """One operator call. ``kind`` is ``"conv"`` or ``"linear"``.

    Conv: x [n, c, h, w], codes [k, c*r*s], y [n, k, oh, ow].
    Linear: x [n, c] (n = batch, c = in features), codes [k, c], y [n, k].
    """

    name: str
    kind: str
    n: int
    c: int
    k: int
    h: int = 1
    w: int = 1
    r: int = 1
    s: int = 1
    stride: int = 1
    pad: int = 0
    bias: bool = False
    x_dist: str = "relu_normal"      # relu_normal | uniform_pm4 | uniform_0_2 | normal
    code_dist: str = "lognormal"     # lognormal | uniform16
    zero_frac: float = 0.10

    @property
    def oh(self) -> int:
        if self.kind == "linear":
            return 1
        return (self.h + 2 * self.pad - self.r) // self.stride + 1

    @property
    def ow(self) -> int:
        if self.kind == "linear":
            return 1
        return (self.w + 2 * self.pad - self.s) // self.stride + 1

    @property
    def crs(self) -> int:
        return self.c * self.r * self.s

    @property
    def x_shape(self) -> tuple:
        if self.kind == "linear":
            return (self.n, self.c)
        return (self.n, self.c, self.h, self.w)

    @property
    def y_shape(self) -> tuple:
        if self.kind == "linear":
            return (self.n, self.k)
        return (self.n, self.k, self.oh, self.ow)

    @property
    def sac(self) -> int:
        """Dense shift-accumulates: one per (output element, reduction term)."""
        return self.n * self.k * self.oh * self.ow * self.crs

    def with_batch(self, n: int) -> "Layer":
        return dataclasses.replace(self, n=n)


def _conv(name, n, c, k, hw, rs, stride, pad, zero_frac):
    return Layer(name, "conv", n=n, c=c, k=k, h=hw, w=hw, r=rs, s=rs,
                 stride=stride, pad=pad, zero_frac=zero_frac)


def resnet18_layers(n: int = 32, zero_frac: float = 0.10) -> list:
    """The 20 convolutions of ResNet-18 (torchvision layout) and its classifier."""
    L = [_conv("conv1", n, 3, 64, 224, 7, 2, 3, zero_frac)]
    for b in range(2):
        for j in (1, 2):
            L.append(_conv(f"layer1.{b}.conv{j}", n, 64, 64, 56, 3, 1, 1, zero_frac))
    cin, hw = 64, 56
    for stage, planes in ((2, 128), (3, 256), (4, 512)):
        L.append(_conv(f"layer{stage}.0.conv1", n, cin, planes, hw, 3, 2, 1, zero_frac))
        L.append(_conv(f"layer{stage}.0.conv2", n, planes, planes, hw // 2, 3, 1, 1, zero_frac))
        L.append(_conv(f"layer{stage}.0.downsample", n, cin, planes, hw, 1, 2, 0, zero_frac))
        for j in (1, 2):
            L.append(_conv(f"layer{stage}.1.conv{j}", n, planes, planes, hw // 2, 3, 1, 1,
                           zero_frac))
        cin, hw = planes, hw // 2
    L.append(Layer("fc", "linear", n=n, c=512, k=1000, bias=True, zero_frac=zero_frac))
    return L


def resnet50_layers(n: int = 128, zero_frac: float = 0.20) -> list:
    """The 53 convolutions of ResNet-50 v1.5 (stride in the 3x3) and its classifier."""
    L = [_conv("conv1", n, 3, 64, 224, 7, 2, 3, zero_frac)]
    cin, hw = 64, 56
    for stage, (planes, blocks) in enumerate(((64, 3), (128, 4), (256, 6), (512, 3)), start=1):
        out = planes * 4
        for b in range(blocks):
            stride = 2 if (b == 0 and stage > 1) else 1
            pre = f"layer{stage}.{b}"
            L.append(_conv(pre + ".conv1", n, cin, planes, hw, 1, 1, 0, zero_frac))
            L.append(_conv(pre + ".conv2", n, planes, planes, hw, 3, stride, 1, zero_frac))
            hw2 = hw // stride
            L.append(_conv(pre + ".conv3", n, planes, out, hw2, 1, 1, 0, zero_frac))
            if b == 0:
                L.append(_conv(pre + ".downsample", n, cin, out, hw, 1, stride, 0, zero_frac))
            cin, hw = out, hw2
    L.append(Layer("fc", "linear", n=n, c=2048, k=1000, bias=True, zero_frac=zero_frac))
    return L


CONFIG_NAMES = {
    0: "linear_b8_256x128",
    1: "conv_n1_c128_28x28_k128_3x3",
    2: "linear_b256_4096x4096",
    3: "resnet18_n32_all_layers",
    4: "resnet50_n128_all_layers",
}
CONFIG_SEEDS = {0: 0, 1: 1, 2: 2, 3: 3, 4: 4}


# Issue-rate probe: a 1 x 1 layer whose weights all have shift 0 (no zero
# weights), 64 MB in and out, 4.3 G add/sub lane-operations: its plan is almost
# only VOP2 adds and subtracts, one load per 64 of them.
VALU_PROBE = Layer("valu_probe", "conv", n=1, c=256, k=256, h=256, w=256, code_dist="shift0",
                   zero_frac=0.0)

# VGG16's fc6 (25088 -> 4096) at batch 1: much generated code for little work,
# where the runtime kernel is the faster path.
LINEAR_25088_B1 = Layer("fc6_b1", "linear", n=1, c=25088, k=4096, bias=True, x_dist="uniform_0_2",
                        zero_frac=0.10)


def config_layers(cfg: int) -> list:
    """Layer list of one benchmark configuration (seed is ``CONFIG_SEEDS[cfg]``)."""
    if cfg == 0:
        return [Layer("linear", "linear", n=8, c=256, k=128, bias=True,
                      x_dist="uniform_pm4", code_dist="uniform16", zero_frac=0.0)]
    if cfg == 1:
        return [_conv("conv3_x", 1, 128, 128, 28, 3, 1, 1, 0.10)]
    if cfg == 2:
        return [Layer("fc6", "linear", n=256, c=4096, k=4096, bias=True,
                      x_dist="uniform_0_2", zero_frac=0.10)]
    if cfg == 3:
        return resnet18_layers(32, 0.10)
    if cfg == 4:
        return resnet50_layers(128, 0.20)
    raise ValueError(f"unknown configuration {cfg}")


# ---------------------------------------------------------------------------
# generators


# Lower bit-width activations (Section 5): fractional bits of each storage width.
# 16 bits are 3.13; 8 bits are 3.5 (3 integer bits with the sign).
ACT_FRAC_BITS = {32: FRAC_BITS, 16: 13, 8: 5}
ACT_DTYPES = {32: np.int32, 16: np.int16, 8: np.int8}


def _fill_chunk(out, start, stop, dist, key, frac=FRAC_BITS):
    rng = np.random.default_rng(key)
    m = stop - start
    if dist == "relu_normal":
        a = rng.standard_normal(m, dtype=np.float32)
        np.abs(a, out=a)
    elif dist == "normal":
        a = rng.standard_normal(m, dtype=np.float32)
    elif dist == "uniform_pm4":
        a = rng.uniform(-4.0, 4.0, m)
    elif dist == "uniform_0_2":
        a = rng.uniform(0.0, 2.0, m)
    else:
        raise ValueError(dist)
    a *= float(1 << frac)
    np.rint(a, out=a)
    if out.dtype != np.int32:  # the narrow formats saturate at their range
        info = np.iinfo(out.dtype)
        np.clip(a, info.min, info.max, out=a)
    out[start:stop] = a


def gen_x(layer: Layer, seed: int, index: int, threads: int | None = None,
          act_bits: int = 32) -> np.ndarray:
    """Activations of ``layer`` as fixed point, seeded by (seed, index): int32 with
    F = 16, or for ``act_bits`` 16 / 8 the same draws as int16 3.13 / int8 3.5,
    saturated at the type's range.

    Chunk ``j`` of the flattened tensor comes from ``default_rng([seed, index, 0, j])``,
    so the result does not depend on the number of threads.
    """
    total = int(np.prod(layer.x_shape))
    out = np.empty(total, dtype=ACT_DTYPES[act_bits])
    frac = ACT_FRAC_BITS[act_bits]
    nchunks = (total + _CHUNK - 1) // _CHUNK
    jobs = [(j * _CHUNK, min(total, (j + 1) * _CHUNK)) for j in range(nchunks)]
    if threads is None:
        threads = min(16, os.cpu_count() or 1)
    if nchunks <= 1 or threads <= 1:
        for j, (a, b) in enumerate(jobs):
            _fill_chunk(out, a, b, layer.x_dist, [seed, index, 0, j], frac)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda jb: _fill_chunk(out, jb[1][0], jb[1][1], layer.x_dist,
                                               [seed, index, 0, jb[0]], frac), enumerate(jobs)))
    return out.reshape(layer.x_shape)


# Shift-code frequencies of weights drawn from N(0, 0.05) and rounded to the nearest
# power of two in the 0..-14 range (code s = weight 2^-s), used as a fixed
# categorical distribution so that generating codes needs no quantisation.
LOGNORMAL_SHIFT_P = np.array([0.0, 1.53744e-12, 0.000406952, 0.0766929, 0.299659, 0.281772,
                              0.166584, 0.0869093, 0.0439207, 0.022019, 0.0110169, 0.00550936,
                              0.00275479, 0.00137741, 0.00137742])


def gen_codes(layer: Layer, seed: int, index: int) -> np.ndarray:
    """Weight codes [k, c*r*s] (uint8, sign << 4 | shift_code), seeded by (seed, index).

    ``uniform16``: sign ~ Bernoulli(1/2), shift code uniform over 0..15.
    ``lognormal``: sign ~ Bernoulli(1/2); shift code drawn from ``LOGNORMAL_SHIFT_P``;
    then each code independently becomes the zero code 15 with probability ``zero_frac``.
    ``shift0``: sign ~ Bernoulli(1/2), every shift 0 and no zero weight (the plan of such
    a layer is one add or subtract per weight and one load per element: an issue-rate
    probe of generated code).
    """
    rng = np.random.default_rng([seed, index, 1])
    shape = (layer.k, layer.crs)
    sign = rng.integers(0, 2, size=shape, dtype=np.uint8)
    if layer.code_dist == "uniform16":
        shift = rng.integers(0, 16, size=shape, dtype=np.uint8)
    elif layer.code_dist == "shift0":
        shift = np.zeros(shape, dtype=np.uint8)
    elif layer.code_dist == "lognormal":
        prob = LOGNORMAL_SHIFT_P / LOGNORMAL_SHIFT_P.sum()
        shift = rng.choice(15, size=shape, p=prob).astype(np.uint8)
        zero = rng.random(shape) < layer.zero_frac
        shift[zero] = 15
    else:
        raise ValueError(layer.code_dist)
    return (sign << 4 | shift).astype(np.uint8)


def gen_bias(layer: Layer, seed: int, index: int):
    """Bias [k] as int32 F=16 from U[-1, 1), or None when the layer has no bias."""
    if not layer.bias:
        return None
    rng = np.random.default_rng([seed, index, 2])
    return np.rint(rng.uniform(-1.0, 1.0, layer.k) * float(1 << FRAC_BITS)).astype(np.int32)


def gen_layer(layer: Layer, seed: int, index: int, threads: int | None = None,
              act_bits: int = 32):
    """(x, codes, bias) for one layer; x of ``act_bits`` bits (see gen_x). The bias keeps
    int32 with the activations' fractional bits."""
    bias = gen_bias(layer, seed, index)
    if bias is not None and act_bits != 32:
        rng = np.random.default_rng([seed, index, 2])
        bias = np.rint(rng.uniform(-1.0, 1.0, layer.k) * float(1 << ACT_FRAC_BITS[act_bits])).astype(np.int32)
    return (gen_x(layer, seed, index, threads, act_bits), gen_codes(layer, seed, index), bias)


def random_codes(rng: np.random.Generator, shape, zero_frac: float = 0.1,
                 max_shift: int = 14) -> np.ndarray:
    """Small-case helper for tests: random sign bits, shift codes uniform over
    0..max_shift, and zero codes (15) with probability ``zero_frac``."""
    sign = rng.integers(0, 2, size=shape, dtype=np.uint8)
    shift = rng.integers(0, max_shift + 1, size=shape, dtype=np.uint8)
    shift[rng.random(shape) < zero_frac] = 15
    return (sign << 4 | shift).astype(np.uint8)


def gen_float_weights(rows: int, cols: int, seed: int) -> np.ndarray:
    """Float32 weights [rows, cols] with Kaiming-normal scale sqrt(2 / cols) (the
    initialisation the paper uses for DeepShift-Q weights; fan-in = cols)."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((rows, cols), dtype=np.float32) * np.float32(np.sqrt(2.0 / cols)))


def gen_ps_params(rows: int, cols: int, seed: int, p_range=(-14.0, 0.0), s_range=(-1.0, 1.0)):
    """DeepShift-PS parameters (P, S) [rows, cols], each uniform over its range (the
    paper initialises both uniformly; the ranges are this project's choice)."""
    rng = np.random.default_rng(seed)
    p = rng.uniform(*p_range, (rows, cols)).astype(np.float32)
    s = rng.uniform(*s_range, (rows, cols)).astype(np.float32)
    return p, s


def gen_float_acts(n: int, seed: int, scale: float = 4.0) -> np.ndarray:
    """Float32 activations [n], normal with standard deviation ``scale``."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(n, dtype=np.float32) * np.float32(scale)


# ---------------------------------------------------------------------------
# ResNet-18 with shift convolutions, chained (the network of the paper's
# Section 6 inference timing). Topology and seeded synthetic parameters only.

BN_SHIFT = 16  # fractional bits of the per-channel batch-normalisation multiplier


def resnet18_graph(n: int = 32) -> list:
    """The forward pass as a list of ops over named int32 buffers (input "x").

    ``conv``: a ResNet-18 convolution layer (``layer``), then batch normalisation,
    the optional residual buffer ``res`` and ReLU when ``relu``: src -> dst.
    ``maxpool``: 3x3, stride 2, pad 1. ``avgpool``: global, [n, c, h, w] -> [n, c].
    ``linear``: the classifier with its bias.
    """
    layers = {L.name: L for L in resnet18_layers(n)}
    g = [{"op": "conv", "layer": layers["conv1"], "src": "x", "dst": "stem", "res": None, "relu": True},
         {"op": "maxpool", "src": "stem", "dst": "b0", "r": 3, "stride": 2, "pad": 1}]
    cur = "b0"
    for stage in (1, 2, 3, 4):
        for b in (0, 1):
            pre = f"layer{stage}.{b}"
            res = cur
            if stage > 1 and b == 0:
                g.append({"op": "conv", "layer": layers[pre + ".downsample"], "src": cur,
                          "dst": pre + ".ds", "res": None, "relu": False})
                res = pre + ".ds"
            g.append({"op": "conv", "layer": layers[pre + ".conv1"], "src": cur, "dst": pre + ".t",
                      "res": None, "relu": True})
            g.append({"op": "conv", "layer": layers[pre + ".conv2"], "src": pre + ".t",
                      "dst": pre + ".out", "res": res, "relu": True})
            cur = pre + ".out"
    g.append({"op": "avgpool", "src": cur, "dst": "pool"})
    g.append({"op": "linear", "layer": layers["fc"], "src": "pool", "dst": "logits"})
    return g


def gen_bn(layer: Layer, seed: int, index: int):
    """Batch-normalisation parameters of a conv layer as (mul [k], add [k]) int32:
    mul = scale * 2**BN_SHIFT with scale = U[0.8, 1.2] / sqrt(C*R*S * E[w^2]) (E[w^2]
    the second moment of the synthetic weight distribution, so that activations
    keep their magnitude from layer to layer), add = N(0, 0.1) * 2**16."""
    rng = np.random.default_rng([seed, index, 3])
    p = LOGNORMAL_SHIFT_P / LOGNORMAL_SHIFT_P.sum()
    ew2 = (1.0 - layer.zero_frac) * float(np.sum(p * 4.0 ** -np.arange(15)))
    scale = rng.uniform(0.8, 1.2, layer.k) / np.sqrt(layer.crs * ew2)
    mul = np.rint(scale * float(1 << BN_SHIFT)).astype(np.int32)
    add = np.rint(rng.normal(0.0, 0.1, layer.k) * float(1 << FRAC_BITS)).astype(np.int32)
    return mul, add


def resnet18_params(n: int = 32, seed: int = 18) -> dict:
    """Seeded synthetic parameters of every layer of ``resnet18_graph(n)``, by layer
    name: codes [k, c*r*s] (uint8), and bn (mul, add) for convs or bias for the fc."""
    params = {}
    for i, L in enumerate(resnet18_layers(n)):
        entry = {"codes": gen_codes(L, seed, i)}
        if L.kind == "conv":
            entry["bn"] = gen_bn(L, seed, i)
        else:
            entry["bias"] = gen_bias(L, seed, i)
        params[L.name] = entry
    return params


def gen_images(n: int, seed: int = 18) -> np.ndarray:
    """Input batch [n, 3, 224, 224] int32 F=16: normalised pixels, N(0, 1) clipped to +-3."""
    rng = np.random.default_rng([seed, 99])
    a = np.clip(rng.standard_normal((n, 3, 224, 224), dtype=np.float32), -3.0, 3.0)
    return np.rint(a * float(1 << FRAC_BITS)).astype(np.int32)
