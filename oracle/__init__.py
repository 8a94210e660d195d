"""Oracle for the DeepShift shift operators -- TEST INFRASTRUCTURE ONLY.

Python access (ctypes, numpy arrays on the host) to the plain-loop C oracle in
``oracle.c``. Only the tests, ``__graft_entry__.smoke()`` and the benchmark's
CPU-baseline leg may import this package; the product library and its Python
binding never do.

Every function takes host numpy arrays in the layouts documented in
``oracle.c``: activations int32 (fixed point, any F), weight codes uint8
(``sign << 4 | shift_code``), optional int32 bias. Activations may also be
int16 or int8 (the lower bit-width formats): they are sign-extended to int32
first, which is their value; every term and sum is then the int32 one.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_DIR = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_DIR, "oracle.c")
_LIB = os.path.join(_DIR, "liboracle.so")
_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int64


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-Wall", "-Wextra", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        lib.oracle_term.restype = ctypes.c_int64
        lib.oracle_term.argtypes = [ctypes.c_int32, ctypes.c_uint8]
        lib.oracle_linear_shift.argtypes = [_P, _P, _P, _P, _I, _I, _I]
        lib.oracle_conv2d_shift.argtypes = [_P, _P, _P, _P] + [_I] * 11
        lib.oracle_conv2d_shift_points.argtypes = [_P, _P, _P] + [_I] * 11 + [_P, _I, _P]
        lib.oracle_linear_shift_points.argtypes = [_P, _P, _P, _I, _I, _I, _P, _I, _P]
        lib.oracle_conv2d_mul.argtypes = [_P, _P, _P, _P] + [_I] * 11
        lib.oracle_linear_shift_backward_data.argtypes = [_P, _P, _P, _I, _I, _I]
        lib.oracle_conv2d_shift_backward_data.argtypes = [_P, _P, _P] + [_I] * 11
        lib.oracle_conv2d_shift_backward_data_points.argtypes = [_P, _P] + [_I] * 11 + [_P, _I, _P]
        lib.oracle_pack_codes.argtypes = [_P, _I, _I, _P]
        lib.oracle_unpack_codes.argtypes = [_P, _I, _I, _P]
        lib.oracle_pack_codes_bits.argtypes = [_P, _I, _I, ctypes.c_int, _P]
        lib.oracle_pack_codes_bits.restype = ctypes.c_int
        lib.oracle_unpack_codes_bits.argtypes = [_P, _I, _I, ctypes.c_int, _P]
        lib.oracle_quantize_q.argtypes = [_P, _I, ctypes.c_int, _P]
        lib.oracle_quantize_ps.argtypes = [_P, _P, _I, ctypes.c_int, _P]
        lib.oracle_to_fixed.argtypes = [_P, _I, ctypes.c_int, _P]
        lib.oracle_epilogue.argtypes = [_P, _I, _I, _I, _P, _P, ctypes.c_int, _P, ctypes.c_int]
        lib.oracle_maxpool2d.argtypes = [_P, _P] + [_I] * 10
        lib.oracle_avgpool_global.argtypes = [_P, _P, _I, _I, _I]
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


def set_threads(n: int) -> None:
    """Number of OpenMP threads the oracle uses (0 = library default)."""
    try:
        omp = ctypes.CDLL("libgomp.so.1")
        if n > 0:
            omp.omp_set_num_threads(ctypes.c_int(n))
    except OSError:
        pass


def max_threads() -> int:
    try:
        omp = ctypes.CDLL("libgomp.so.1")
        return int(omp.omp_get_max_threads())
    except OSError:
        return 1


def term(x: int, code: int) -> int:
    """flip(floor(x * 2**-shift), sign) for one activation and one code."""
    return int(_load().oracle_term(int(x), int(code)))


def linear_shift(x, codes, bias=None):
    """LinearShift: x [batch, in] int32, codes [out, in] uint8 -> y [batch, out] int32."""
    x = _c(x, np.int32); codes = _c(codes, np.uint8); bias = _c(bias, np.int32)
    batch, fin = x.shape
    fout, fin2 = codes.shape
    assert fin == fin2 and (bias is None or bias.shape == (fout,))
    y = np.empty((batch, fout), np.int32)
    _load().oracle_linear_shift(_ptr(x), _ptr(codes), _ptr(bias), _ptr(y), batch, fin, fout)
    return y


def out_size(h, pad, r, stride):
    return (h + 2 * pad - r) // stride + 1


def conv2d_shift(x, codes, bias=None, r=3, s=None, stride=1, pad=0):
    """ConvShift: x [N, C, H, W] int32, codes [K, C*R*S] uint8 -> y [N, K, OH, OW].

    ``stride`` and ``pad`` are ints or (h, w) pairs.
    """
    s = r if s is None else s
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    x = _c(x, np.int32); codes = _c(codes, np.uint8); bias = _c(bias, np.int32)
    N, C, H, W = x.shape
    K = codes.shape[0]
    assert codes.shape == (K, C * r * s) or codes.shape == (K, C, r, s)
    OH, OW = out_size(H, ph, r, sh), out_size(W, pw, s, sw)
    y = np.empty((N, K, OH, OW), np.int32)
    _load().oracle_conv2d_shift(_ptr(x), _ptr(codes), _ptr(bias), _ptr(y),
                                N, C, H, W, K, r, s, sh, sw, ph, pw)
    return y


def conv2d_shift_points(x, codes, bias, idx, r=3, s=None, stride=1, pad=0):
    """Selected outputs y.flat[idx] of ``conv2d_shift`` (idx int64 flat indices)."""
    s = r if s is None else s
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    x = _c(x, np.int32); codes = _c(codes, np.uint8); bias = _c(bias, np.int32)
    idx = _c(idx, np.int64)
    N, C, H, W = x.shape
    K = codes.shape[0]
    out = np.empty(idx.shape, np.int32)
    _load().oracle_conv2d_shift_points(_ptr(x), _ptr(codes), _ptr(bias), N, C, H, W, K, r, s,
                                       sh, sw, ph, pw, _ptr(idx), idx.size, _ptr(out))
    return out


def linear_shift_points(x, codes, bias, idx):
    """Selected outputs y.flat[idx] of ``linear_shift``."""
    x = _c(x, np.int32); codes = _c(codes, np.uint8); bias = _c(bias, np.int32)
    idx = _c(idx, np.int64)
    batch, fin = x.shape
    out = np.empty(idx.shape, np.int32)
    _load().oracle_linear_shift_points(_ptr(x), _ptr(codes), _ptr(bias), batch, fin,
                                       codes.shape[0], _ptr(idx), idx.size, _ptr(out))
    return out


def linear_shift_backward_data(dy, codes):
    """Input gradient of LinearShift: dy [batch, out] int32, codes [out, in] uint8 ->
    dx [batch, in] = sum_o term(dy[b, o], code[o, i])."""
    dy = _c(dy, np.int32); codes = _c(codes, np.uint8)
    batch, fout = dy.shape
    fout2, fin = codes.shape
    assert fout == fout2
    dx = np.empty((batch, fin), np.int32)
    _load().oracle_linear_shift_backward_data(_ptr(dy), _ptr(codes), _ptr(dx), batch, fin, fout)
    return dx


def conv2d_shift_backward_data(dy, codes, x_shape, r=3, s=None, stride=1, pad=0):
    """Input gradient of ConvShift: dy [N, K, OH, OW] int32, codes [K, C*R*S] ->
    dx of the forward input's shape x_shape = (N, C, H, W)."""
    s = r if s is None else s
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    dy = _c(dy, np.int32); codes = _c(codes, np.uint8)
    N, C, H, W = x_shape
    K = codes.shape[0]
    assert dy.shape == (N, K, out_size(H, ph, r, sh), out_size(W, pw, s, sw))
    assert codes.size == K * C * r * s
    dx = np.empty((N, C, H, W), np.int32)
    _load().oracle_conv2d_shift_backward_data(_ptr(dy), _ptr(codes), _ptr(dx), N, C, H, W, K, r, s,
                                              sh, sw, ph, pw)
    return dx


def conv2d_shift_backward_data_points(dy, codes, x_shape, idx, r=3, s=None, stride=1, pad=0):
    """Selected elements dx.flat[idx] of ``conv2d_shift_backward_data``, each gathered alone."""
    s = r if s is None else s
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    dy = _c(dy, np.int32); codes = _c(codes, np.uint8); idx = _c(idx, np.int64)
    N, C, H, W = x_shape
    K = codes.shape[0]
    out = np.empty(idx.shape, np.int32)
    _load().oracle_conv2d_shift_backward_data_points(_ptr(dy), _ptr(codes), N, C, H, W, K, r, s,
                                                     sh, sw, ph, pw, _ptr(idx), idx.size, _ptr(out))
    return out


def conv2d_mul(x, wts, bias=None, r=3, s=None, stride=1, pad=0):
    """Multiplication-based comparison: y = wrap32(b + sum x*w), int32 weights [K, C*R*S]."""
    s = r if s is None else s
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    x = _c(x, np.int32); wts = _c(wts, np.int32); bias = _c(bias, np.int32)
    N, C, H, W = x.shape
    K = wts.shape[0]
    OH, OW = out_size(H, ph, r, sh), out_size(W, pw, s, sw)
    y = np.empty((N, K, OH, OW), np.int32)
    _load().oracle_conv2d_mul(_ptr(x), _ptr(wts), _ptr(bias), _ptr(y), N, C, H, W, K, r, s,
                              sh, sw, ph, pw)
    return y


def sext24(a):
    """Each int32 element's low 24 bits taken as a signed 24-bit value (int32)."""
    a = np.asarray(a, dtype=np.int32)
    return ((a.astype(np.int64) & 0xFFFFFF) ^ 0x800000).astype(np.int64) - 0x800000


def conv2d_mul24(x, wts, bias=None, r=3, s=None, stride=1, pad=0):
    """The 24-bit multiplication comparison: conv2d_mul of the operands' low 24
    bits as signed values (what a v_mad_i32_i24 per term computes)."""
    return conv2d_mul(sext24(x).astype(np.int32), sext24(wts).astype(np.int32), bias, r=r, s=s,
                      stride=stride, pad=pad)


def pack_codes(codes):
    """codes [rows, cols] uint8 -> packed [rows, ceil(cols/6)] uint32."""
    codes = _c(codes, np.uint8)
    rows, cols = codes.shape
    out = np.empty((rows, (cols + 5) // 6), np.uint32)
    _load().oracle_pack_codes(_ptr(codes), rows, cols, _ptr(out))
    return out


def unpack_codes(packed, cols):
    packed = _c(packed, np.uint32)
    rows = packed.shape[0]
    out = np.empty((rows, cols), np.uint8)
    _load().oracle_unpack_codes(_ptr(packed), rows, cols, _ptr(out))
    return out


def pack_codes_bits(codes, bits):
    """codes [rows, cols] uint8 (5-bit form) -> words of `bits`-bit codes, floor(32 / bits)
    per word; None when a shift does not fit."""
    codes = _c(codes, np.uint8)
    rows, cols = codes.shape
    per = 32 // bits
    out = np.zeros((rows, (cols + per - 1) // per), np.uint32)
    if _load().oracle_pack_codes_bits(_ptr(codes), rows, cols, int(bits), _ptr(out)) != 0:
        return None
    return out


def unpack_codes_bits(packed, cols, bits):
    packed = _c(packed, np.uint32)
    rows = packed.shape[0]
    out = np.empty((rows, cols), np.uint8)
    _load().oracle_unpack_codes_bits(_ptr(packed), rows, cols, int(bits), _ptr(out))
    return out


def quantize_q(w, max_shift=14):
    """DeepShift-Q codes of float32 weights (any shape): sign(w), round(log2|w|) clipped
    to -max_shift .. 0."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    out = np.empty(w.shape, np.uint8)
    _load().oracle_quantize_q(_ptr(w), w.size, int(max_shift), _ptr(out))
    return out


def quantize_ps(P, S, max_shift=14):
    """DeepShift-PS codes from float32 shift and sign parameters of the same shape."""
    P = np.ascontiguousarray(P, dtype=np.float32)
    S = np.ascontiguousarray(S, dtype=np.float32)
    assert P.shape == S.shape
    out = np.empty(P.shape, np.uint8)
    _load().oracle_quantize_ps(_ptr(P), _ptr(S), P.size, int(max_shift), _ptr(out))
    return out


def to_fixed(x, frac_bits=16):
    """round(x * 2**F), halves away from zero, saturated to int32 (NaN -> 0)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.int32)
    _load().oracle_to_fixed(_ptr(x), x.size, int(frac_bits), _ptr(out))
    return out


def to_fixed_narrow(x, frac_bits, bits):
    """round(x * 2^frac_bits) (halves away from zero, NaN -> 0) saturated to a signed
    integer of `bits` bits (16 or 8): the int32 rounding of ``to_fixed``, clamped to the
    narrower range (which lies inside int32, so the clamp of the int32-saturated value
    is the clamp of the exact one)."""
    lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    dt = {16: np.int16, 8: np.int8}[bits]
    return np.clip(to_fixed(x, frac_bits).astype(np.int64), lo, hi).astype(dt)


def epilogue(y, mul=None, add=None, mul_shift=16, residual=None, relu=False):
    """Copy of y [N, K, ...] after the fused epilogue: affine (mul, add per channel,
    floor(v * mul / 2**mul_shift) + add), + residual, ReLU; int32 wrap-around."""
    y = np.array(y, dtype=np.int32, copy=True, order="C")
    N, K = y.shape[0], y.shape[1]
    P = int(np.prod(y.shape[2:])) if y.ndim > 2 else 1
    mul = _c(mul, np.int32); add = _c(add, np.int32); residual = _c(residual, np.int32)
    assert residual is None or residual.shape == y.shape
    _load().oracle_epilogue(_ptr(y), N, K, P, _ptr(mul), _ptr(add), int(mul_shift),
                            _ptr(residual), int(bool(relu)))
    return y


def maxpool2d(x, r=3, s=None, stride=2, pad=1):
    """Max pooling of x [N, C, H, W] (int32); padding positions are ignored."""
    s = r if s is None else s
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    x = _c(x, np.int32)
    N, C, H, W = x.shape
    y = np.empty((N, C, out_size(H, ph, r, sh), out_size(W, pw, s, sw)), np.int32)
    _load().oracle_maxpool2d(_ptr(x), _ptr(y), N, C, H, W, r, s, sh, sw, ph, pw)
    return y


def avgpool_global(x):
    """x [N, C, H, W] -> [N, C]: floor(sum over H*W / (H*W))."""
    x = _c(x, np.int32)
    N, C = x.shape[:2]
    HW = int(np.prod(x.shape[2:]))
    y = np.empty((N, C), np.int32)
    _load().oracle_avgpool_global(_ptr(x), _ptr(y), N, C, HW)
    return y


def network_forward(graph, params, x, mul_shift=16, keep=False):
    """Runs a graph of ops (see ``workloads.resnet18_graph``) on x with the oracle:
    conv -> ConvShift, then the epilogue with the layer's batch normalisation
    (mul, add), the residual buffer and ReLU; maxpool; global avgpool; linear ->
    LinearShift with bias. Returns the last op's output (all buffers if keep)."""
    buf = {"x": np.ascontiguousarray(x, dtype=np.int32)}
    out = None
    for op in graph:
        kind = op["op"]
        src = buf[op["src"]]
        if kind == "conv":
            L = op["layer"]
            p = params[L.name]
            y = conv2d_shift(src, p["codes"], None, r=L.r, s=L.s, stride=L.stride, pad=L.pad)
            mul, add = p["bn"]
            res = buf[op["res"]] if op["res"] else None
            out = epilogue(y, mul, add, mul_shift, residual=res, relu=op["relu"])
        elif kind == "maxpool":
            out = maxpool2d(src, r=op["r"], stride=op["stride"], pad=op["pad"])
        elif kind == "avgpool":
            out = avgpool_global(src)
        elif kind == "linear":
            L = op["layer"]
            p = params[L.name]
            out = linear_shift(src, p["codes"], p["bias"])
        else:
            raise ValueError(kind)
        buf[op["dst"]] = out
    return buf if keep else out
