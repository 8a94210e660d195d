"""PyTorch-facing wrappers of the C ABI.

PyTorch provides the device memory and the stream; every computation runs in
the HIP library. Tensors must be contiguous int32 CUDA (ROCm) tensors; packed
weights are int32 tensors holding the uint32 words bit for bit.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from ._native import DeepShiftError, call, lib

__all__ = ["DeepShiftError", "code_bits_flag", "describe_conv2d", "packed_row_words", "pack_shift_weights", "unpack_shift_weights",
           "linear_shift", "conv2d_shift", "linear_mul_i32", "conv2d_mul_i32", "out_size",
           "quantize_shift_weights_q", "quantize_shift_weights_q_many", "quantize_shift_weights_ps",
           "to_fixed_point", "conv2d_shift_fused", "maxpool2d", "avgpool2d_global", "DS_RELU",
           "DS_JIT_RESIDUAL", "JitConv", "jit_conv_image", "conv2d_shift_backward_data",
           "linear_shift_backward_data", "describe_conv2d_backward_data", "JitConvBackwardData",
           "layer_plan", "run_layer_plan", "set_tuning", "get_tuning", "tuning", "DS_MUL_I24",
           "JitConvMul", "jit_conv_mul_image", "DS_ACT_I16", "DS_ACT_I8", "act_bits_flag"]

DS_RELU = 1


def code_bits_flag(bits: int) -> int:
    """The DS_CODE_BITS flags field for packed codes of `bits` bits (0 for the default 5)."""
    if bits not in (2, 3, 4, 5):
        raise ValueError("code bits must be 2..5")
    return 0 if bits == 5 else bits << 8


def packed_row_words(cols: int, bits: int = 5) -> int:
    return int(lib().ds_packed_row_words_bits(int(cols), int(bits)))


def pack_shift_weights(codes, bits: int = 5) -> np.ndarray:
    """Host codes [rows, cols] (uint8, sign << 4 | shift) -> packed words
    [rows, ceil(cols / floor(32 / bits))] of `bits`-bit codes (5: six per word)."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    if codes.ndim != 2:
        codes = codes.reshape(codes.shape[0], -1)
    rows, cols = codes.shape
    out = np.empty((rows, max(packed_row_words(cols, bits), 0)), dtype=np.uint32)
    call("ds_pack_shift_weights_bits", codes.ctypes.data, rows, cols, bits, out.ctypes.data, out.size)
    return out


def unpack_shift_weights(packed, cols: int, bits: int = 5) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint32)
    rows = packed.shape[0]
    out = np.empty((rows, cols), dtype=np.uint8)
    call("ds_unpack_shift_weights_bits", packed.ctypes.data, rows, cols, bits, out.ctypes.data, out.size)
    return out


def describe_conv2d(n, c, h, w, k, kernel_size, stride=1, padding=0) -> str:
    """Name of the kernel the library runs for this ConvShift shape (LinearShift:
    a 1x1 convolution with h = w = 1)."""
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    import ctypes
    buf = ctypes.create_string_buffer(128)
    call("ds_conv2d_shift_describe", n, c, h, w, k, r, s, sh, sw, ph, pw, buf, len(buf))
    return buf.value.decode()


def describe_conv2d_backward_data(n, c, h, w, k, kernel_size, stride=1, padding=0) -> str:
    """What the library runs for the input gradient of this forward ConvShift shape."""
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    import ctypes
    buf = ctypes.create_string_buffer(512)
    call("ds_conv2d_shift_backward_data_describe", n, c, h, w, k, r, s, sh, sw, ph, pw, buf, len(buf))
    return buf.value.decode()


DS_ACT_I16 = 1 << 12
DS_ACT_I8 = 2 << 12
_ACT_DTYPES = {32: torch.int32, 16: torch.int16, 8: torch.int8}


def act_bits_flag(bits: int) -> int:
    """The DS_ACT_* flags field for activations of `bits` bits (32, 16 or 8)."""
    if bits not in _ACT_DTYPES:
        raise ValueError("activation bits must be 32, 16 or 8")
    return {32: 0, 16: DS_ACT_I16, 8: DS_ACT_I8}[bits]


def _dev_int(t: torch.Tensor, name: str, bits: int) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != _ACT_DTYPES[bits] and not (bits == 32 and t.dtype == torch.uint32):
        raise TypeError(f"{name} must be {_ACT_DTYPES[bits]}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _dev_i32(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype not in (torch.int32, torch.uint32):
        raise TypeError(f"{name} must be int32, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _dev_f32(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def out_size(size: int, pad: int, k: int, stride: int) -> int:
    return (size + 2 * pad - k) // stride + 1


def _pair(v):
    return (int(v), int(v)) if np.isscalar(v) else (int(v[0]), int(v[1]))


def linear_shift(x: torch.Tensor, w_packed: torch.Tensor, bias: torch.Tensor | None = None,
                 frac_bits: int = 16, out: torch.Tensor | None = None, relu: bool = False,
                 code_bits: int = 5) -> torch.Tensor:
    """LinearShift: y[b, o] = bias[o] + sum_i term(x[b, i], code[o, i]) (int32, mod 2^32),
    then max(y, 0) when relu."""
    _dev_i32(x, "x"); _dev_i32(w_packed, "w_packed")
    if bias is not None:
        _dev_i32(bias, "bias")
    batch, fin = x.shape
    fout = w_packed.shape[0]
    y = out if out is not None else torch.empty((batch, fout), dtype=torch.int32, device=x.device)
    _dev_i32(y, "out")
    with torch.cuda.device(x.device):
        call("ds_linear_shift", _ptr(x), _ptr(w_packed), _ptr(bias), _ptr(y), batch, fin, fout,
             frac_bits, (DS_RELU if relu else 0) | code_bits_flag(code_bits), _stream(x.device))
    return y


def conv2d_shift(x: torch.Tensor, w_packed: torch.Tensor, bias: torch.Tensor | None,
                 kernel_size, stride=1, padding=0, frac_bits: int = 16,
                 out: torch.Tensor | None = None, relu: bool = False,
                 code_bits: int = 5) -> torch.Tensor:
    """ConvShift (NCHW): y[n, k, oh, ow] = bias[k] + sum_{c,r,s} term(x[...], code[k, c, r, s]),
    then max(y, 0) when relu."""
    _dev_i32(x, "x"); _dev_i32(w_packed, "w_packed")
    if bias is not None:
        _dev_i32(bias, "bias")
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    n, c, h, w = x.shape
    k = w_packed.shape[0]
    oh, ow = out_size(h, ph, r, sh), out_size(w, pw, s, sw)
    y = out if out is not None else torch.empty((n, k, max(oh, 0), max(ow, 0)), dtype=torch.int32,
                                                device=x.device)
    _dev_i32(y, "out")
    with torch.cuda.device(x.device):
        call("ds_conv2d_shift", _ptr(x), _ptr(w_packed), _ptr(bias), _ptr(y), n, c, h, w, k, r, s,
             sh, sw, ph, pw, frac_bits, (DS_RELU if relu else 0) | code_bits_flag(code_bits),
             _stream(x.device))
    return y


def conv2d_shift_backward_data(dy: torch.Tensor, w_packed: torch.Tensor, x_shape, kernel_size,
                               stride=1, padding=0, frac_bits: int = 16,
                               out: torch.Tensor | None = None, code_bits: int = 5) -> torch.Tensor:
    """Input gradient of a ConvShift layer (NCHW): dx[n, c, ih, iw] = sum of
    term(dy[n, k, oh, ow], code[k, c, r, s]) over the forward connections. x_shape =
    (n, c, h, w) of the forward input; dy has the forward output's shape."""
    _dev_i32(dy, "dy"); _dev_i32(w_packed, "w_packed")
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    n, c, h, w = (int(v) for v in x_shape)
    k = w_packed.shape[0]
    dx = out if out is not None else torch.empty((n, c, h, w), dtype=torch.int32, device=dy.device)
    _dev_i32(dx, "out")
    with torch.cuda.device(dy.device):
        call("ds_conv2d_shift_backward_data", _ptr(dy), _ptr(w_packed), _ptr(dx), n, c, h, w, k, r, s,
             sh, sw, ph, pw, frac_bits, code_bits_flag(code_bits), _stream(dy.device))
    return dx


def linear_shift_backward_data(dy: torch.Tensor, w_packed: torch.Tensor, in_features: int,
                               frac_bits: int = 16, out: torch.Tensor | None = None,
                               code_bits: int = 5) -> torch.Tensor:
    """Input gradient of a LinearShift layer: dx[b, i] = sum_o term(dy[b, o], code[o, i])."""
    _dev_i32(dy, "dy"); _dev_i32(w_packed, "w_packed")
    batch, fout = dy.shape
    dx = out if out is not None else torch.empty((batch, in_features), dtype=torch.int32, device=dy.device)
    _dev_i32(dx, "out")
    with torch.cuda.device(dy.device):
        call("ds_linear_shift_backward_data", _ptr(dy), _ptr(w_packed), _ptr(dx), batch, in_features,
             fout, frac_bits, code_bits_flag(code_bits), _stream(dy.device))
    return dx


DS_MUL_I24 = 4


def linear_mul_i32(x, w, bias=None, out=None, mul24: bool = False):
    """Multiplication-based comparison: y = bias + x @ w.T (int32, mod 2^32); with
    mul24 each product takes the low 24 bits of both operands as signed values."""
    _dev_i32(x, "x"); _dev_i32(w, "w")
    batch, fin = x.shape
    fout = w.shape[0]
    y = out if out is not None else torch.empty((batch, fout), dtype=torch.int32, device=x.device)
    with torch.cuda.device(x.device):
        call("ds_linear_mul_i32", _ptr(x), _ptr(w), _ptr(bias), _ptr(y), batch, fin, fout,
             DS_MUL_I24 if mul24 else 0, _stream(x.device))
    return y


def conv2d_mul_i32(x, w, bias, kernel_size, stride=1, padding=0, out=None, mul24: bool = False):
    """Multiplication-based comparison convolution with int32 weights [K, C*R*S]; with
    mul24 each product takes the low 24 bits of both operands as signed values."""
    _dev_i32(x, "x"); _dev_i32(w, "w")
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    n, c, h, wd = x.shape
    k = w.shape[0]
    oh, ow = out_size(h, ph, r, sh), out_size(wd, pw, s, sw)
    y = out if out is not None else torch.empty((n, k, oh, ow), dtype=torch.int32, device=x.device)
    with torch.cuda.device(x.device):
        call("ds_conv2d_mul_i32", _ptr(x), _ptr(w), _ptr(bias), _ptr(y), n, c, h, wd, k, r, s,
             sh, sw, ph, pw, DS_MUL_I24 if mul24 else 0, _stream(x.device))
    return y


def _weight_rows(t: torch.Tensor):
    rows = t.shape[0]
    return rows, (t.numel() // rows if rows else 0)


def quantize_shift_weights_q(w: torch.Tensor, max_shift: int = 14,
                             out: torch.Tensor | None = None, code_bits: int = 5) -> torch.Tensor:
    """DeepShift-Q: float32 weights [rows, ...] -> packed codes [rows, words] (int32 bits),
    `code_bits`-bit codes (max_shift at most 2^(code_bits-1) - 2)."""
    _dev_f32(w, "w")
    rows, cols = _weight_rows(w)
    y = out if out is not None else torch.empty((rows, max(packed_row_words(cols, code_bits), 0)),
                                                dtype=torch.int32, device=w.device)
    _dev_i32(y, "out")
    with torch.cuda.device(w.device):
        call("ds_quantize_shift_weights_q", _ptr(w), rows, cols, max_shift, _ptr(y),
             code_bits_flag(code_bits), _stream(w.device))
    return y


def quantize_shift_weights_q_many(ws, max_shift: int = 14, outs=None, code_bits: int = 5) -> list:
    """DeepShift-Q for a list of float32 weight tensors in one library call."""
    import ctypes
    if not ws:
        raise ValueError("no tensors")
    for i, w in enumerate(ws):
        _dev_f32(w, f"ws[{i}]")
    shapes = [_weight_rows(w) for w in ws]
    if outs is None:
        outs = [torch.empty((r, max(packed_row_words(c, code_bits), 0)), dtype=torch.int32, device=w.device)
                for w, (r, c) in zip(ws, shapes)]
    for i, o in enumerate(outs):
        _dev_i32(o, f"outs[{i}]")
    n = len(ws)
    wp = (ctypes.c_void_p * n)(*[w.data_ptr() for w in ws])
    op = (ctypes.c_void_p * n)(*[o.data_ptr() for o in outs])
    rows = (ctypes.c_int64 * n)(*[r for r, _ in shapes])
    cols = (ctypes.c_int64 * n)(*[c for _, c in shapes])
    dev = ws[0].device
    with torch.cuda.device(dev):
        call("ds_quantize_shift_weights_q_many", n, wp, rows, cols, max_shift, op,
             code_bits_flag(code_bits), _stream(dev))
    return outs


def quantize_shift_weights_ps(p: torch.Tensor, s: torch.Tensor, max_shift: int = 14,
                              out: torch.Tensor | None = None, code_bits: int = 5) -> torch.Tensor:
    """DeepShift-PS: shift and sign parameters [rows, ...] -> packed codes [rows, words]."""
    _dev_f32(p, "p"); _dev_f32(s, "s")
    if p.shape != s.shape:
        raise ValueError("p and s must have the same shape")
    rows, cols = _weight_rows(p)
    y = out if out is not None else torch.empty((rows, max(packed_row_words(cols, code_bits), 0)),
                                                dtype=torch.int32, device=p.device)
    _dev_i32(y, "out")
    with torch.cuda.device(p.device):
        call("ds_quantize_shift_weights_ps", _ptr(p), _ptr(s), rows, cols, max_shift, _ptr(y),
             code_bits_flag(code_bits), _stream(p.device))
    return y


def to_fixed_point(x: torch.Tensor, frac_bits: int = 16,
                   out: torch.Tensor | None = None, bits: int = 32) -> torch.Tensor:
    """round(x * 2**frac_bits), halves away from zero, saturated to a signed integer of
    `bits` bits (32, or 16 / 8 for the lower bit-width activations)."""
    _dev_f32(x, "x")
    y = out if out is not None else torch.empty(x.shape, dtype=_ACT_DTYPES[bits], device=x.device)
    _dev_int(y, "out", bits)
    with torch.cuda.device(x.device):
        call("ds_to_fixed_point", _ptr(x), x.numel(), frac_bits, _ptr(y), act_bits_flag(bits),
             _stream(x.device))
    return y


def conv2d_shift_fused(x: torch.Tensor, w_packed: torch.Tensor, bias, kernel_size, stride=1,
                       padding=0, mul=None, add=None, mul_shift: int = 16, residual=None,
                       relu: bool = False, frac_bits: int = 16, out=None,
                       code_bits: int = 5) -> torch.Tensor:
    """ConvShift, then per channel floor(v * mul / 2**mul_shift) + add, + residual, ReLU."""
    _dev_i32(x, "x"); _dev_i32(w_packed, "w_packed")
    for t, name in ((bias, "bias"), (mul, "mul"), (add, "add"), (residual, "residual")):
        if t is not None:
            _dev_i32(t, name)
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    n, c, h, w = x.shape
    k = w_packed.shape[0]
    oh, ow = out_size(h, ph, r, sh), out_size(w, pw, s, sw)
    y = out if out is not None else torch.empty((n, k, max(oh, 0), max(ow, 0)), dtype=torch.int32,
                                                device=x.device)
    _dev_i32(y, "out")
    with torch.cuda.device(x.device):
        call("ds_conv2d_shift_fused", _ptr(x), _ptr(w_packed), _ptr(bias), _ptr(mul), _ptr(add),
             mul_shift, _ptr(residual), _ptr(y), n, c, h, w, k, r, s, sh, sw, ph, pw, frac_bits,
             (DS_RELU if relu else 0) | code_bits_flag(code_bits), _stream(x.device))
    return y


def maxpool2d(x: torch.Tensor, kernel_size=3, stride=2, padding=1, out=None) -> torch.Tensor:
    """Max pooling (int32 NCHW); padding positions are ignored."""
    _dev_i32(x, "x")
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    n, c, h, w = x.shape
    oh, ow = out_size(h, ph, r, sh), out_size(w, pw, s, sw)
    y = out if out is not None else torch.empty((n, c, max(oh, 0), max(ow, 0)), dtype=torch.int32,
                                                device=x.device)
    _dev_i32(y, "out")
    with torch.cuda.device(x.device):
        call("ds_maxpool2d", _ptr(x), _ptr(y), n, c, h, w, r, s, sh, sw, ph, pw, 0, _stream(x.device))
    return y


def avgpool2d_global(x: torch.Tensor, out=None) -> torch.Tensor:
    """x [n, c, h, w] -> [n, c]: floor of the mean over h*w."""
    _dev_i32(x, "x")
    n, c, h, w = x.shape
    y = out if out is not None else torch.empty((n, c), dtype=torch.int32, device=x.device)
    _dev_i32(y, "out")
    with torch.cuda.device(x.device):
        call("ds_avgpool2d_global", _ptr(x), _ptr(y), n, c, h, w, 0, _stream(x.device))
    return y


DS_JIT_RESIDUAL = 2


def _host_i32(a, k, name):
    if a is None:
        return None
    a = np.ascontiguousarray(a.cpu().numpy() if isinstance(a, torch.Tensor) else a)
    if a.dtype != np.int32 or a.size != k:
        raise ValueError(f"{name} must be {k} int32 values")
    return a


def _jit_args(w_packed, k, bias, mul, add):
    wp = np.ascontiguousarray(w_packed.cpu().numpy() if isinstance(w_packed, torch.Tensor) else w_packed)
    wp = wp.view(np.uint32) if wp.dtype in (np.int32, np.uint32) else wp
    if wp.dtype != np.uint32 or wp.ndim != 2 or wp.shape[0] != k:
        raise ValueError("w_packed must be packed words [k][row_words]")
    return wp, _host_i32(bias, k, "bias"), _host_i32(mul, k, "mul"), _host_i32(add, k, "add")


def _np_ptr(a):
    return None if a is None else a.ctypes.data


def jit_conv_image(w_packed, x_shape, kernel_size, stride=1, padding=0, bias=None, mul=None,
                   add=None, mul_shift: int = 16, residual: bool = False, relu: bool = False,
                   splits: int = 0, code_bits: int = 5, act_bits: int = 32) -> bytes:
    """The code object a JitConv with these arguments would load (host only)."""
    k = int(w_packed.shape[0])
    wp, b, m, a = _jit_args(w_packed, k, bias, mul, add)
    n, c, h, w = x_shape
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    flags = (DS_RELU if relu else 0) | (DS_JIT_RESIDUAL if residual else 0) | code_bits_flag(code_bits) \
        | act_bits_flag(act_bits)
    size = ctypes.c_int64(0)
    args = [_np_ptr(wp), _np_ptr(b), _np_ptr(m), _np_ptr(a), mul_shift, n, c, h, w, k, r, s, sh, sw,
            ph, pw, flags, splits]
    st = lib().ds_jit_conv_image(*args, None, 0, ctypes.byref(size))
    if st not in (0, 4):
        call("ds_jit_conv_image", *args, None, 0, ctypes.byref(size))
    buf = ctypes.create_string_buffer(size.value)
    call("ds_jit_conv_image", *args, buf, size.value, ctypes.byref(size))
    return buf.raw[:size.value]


class JitConv:
    """A weight-specialised ConvShift (``ds_jit_conv_*``): machine code generated
    for fixed weights and a fixed input shape, loaded on the current device.

    ``w_packed``, ``bias``, ``mul`` and ``add`` may be host arrays or tensors (they
    are read on the host while the code is generated)."""

    def __init__(self, w_packed, x_shape, kernel_size, stride=1, padding=0, bias=None, mul=None,
                 add=None, mul_shift: int = 16, residual: bool = False, relu: bool = False,
                 splits: int = 0, device="cuda:0", code_bits: int = 5, act_bits: int = 32):
        self.k = int(w_packed.shape[0])
        wp, b, m, a = _jit_args(w_packed, self.k, bias, mul, add)
        self.x_shape = tuple(int(v) for v in x_shape)
        n, c, h, w = self.x_shape
        r, s = _pair(kernel_size)
        sh, sw = _pair(stride)
        ph, pw = _pair(padding)
        self.y_shape = (n, self.k, out_size(h, ph, r, sh), out_size(w, pw, s, sw))
        self.device = torch.device(device)
        self.residual = residual
        self.act_bits = act_bits
        flags = (DS_RELU if relu else 0) | (DS_JIT_RESIDUAL if residual else 0) | code_bits_flag(code_bits) \
            | act_bits_flag(act_bits)
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            call("ds_jit_conv_create", _np_ptr(wp), _np_ptr(b), _np_ptr(m), _np_ptr(a), mul_shift,
                 n, c, h, w, self.k, r, s, sh, sw, ph, pw, flags, splits, ctypes.byref(handle))
        self._h = handle
        self._query()
        self.crs = c * r * s
        self.out_pixels, self.out_channels = n * self.y_shape[2] * self.y_shape[3], self.k
        self.sac = self.out_pixels * self.k * self.crs
        self.linear = h == w == r == s == 1 and ph == pw == 0

    def _query(self):
        cb, seg, sp = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
        call("ds_jit_conv_query", self._h, ctypes.byref(cb), ctypes.byref(seg), ctypes.byref(sp))
        self.code_bytes, self.segments, self.splits = cb.value, seg.value, sp.value
        tn, ws, pg, tiles, tr = (ctypes.c_int32() for _ in range(5))
        call("ds_jit_conv_layout", self._h, ctypes.byref(tn), ctypes.byref(ws), ctypes.byref(pg),
             ctypes.byref(tiles), ctypes.byref(tr))
        # Output channels per segment, waves per 64 pixels (each streaming code of
        # its own), groups of 64 pixels per workgroup, the pixel tiles (workgroups)
        # that run each segment, and whether a LinearShift runs on x^T.
        self.channels, self.wsplit, self.pixel_groups, self.pixel_tiles = tn.value, ws.value, pg.value, tiles.value
        self.transposed = bool(tr.value)

    # Cost model of the two paths on MI355X (microseconds), fitted to calls timed
    # back to back. A plan's waves each stream their share of the straight-line
    # code at about 1.6 GB/s when few waves share it (instruction fetch: a 64-byte
    # line per L2 round trip with a few in flight; the 4096 -> 4096 LinearShift
    # at batch 256, 290 KB per wave, 174 us), and the chip issues at most 0.355
    # wave-instructions per SIMD per clock (872 G/s: the ResNet-50 plans, whose
    # waves share their code, and a probe of adds). Code words are about 1.05 per
    # instruction; each share's code runs once per group of 64 pixels (a pixel
    # tile holds 1, 2 or 4 of them).
    # Launch and set-up add about 3 us, a split reduction (fill pass, atomics) 3
    # us more. The runtime kernel decodes its weights and launches 2-5 kernels per
    # call (about 25 us for a convolution, 40 us for a LinearShift at 256 rows or
    # more, whose operands it transposes), then runs at up to 15 T dense SACs/s
    # on full tiles of 256 output pixels (a ragged last tile wastes its lanes),
    # reading its packed weights at 4 TB/s. A LinearShift of fewer than 256 rows
    # takes the small-batch kernel instead (lanes own output channels): about 6
    # us plus 9.6 T dense SACs/s, or its packed weights at 1.75 TB/s when they
    # dominate (batch 1: each code decoded for one row). A LinearShift plan on x^T adds its
    # two transposing passes and runs its kernel about 15 % slower than modelled
    # (2.5 us + 1.16 x the plan's own estimate fits batches 64-256 within 15 %).
    PLAN_STREAM_BPUS = 1.6e3        # code bytes per us per wave
    PLAN_ISSUE_PER_US = 872e3       # wave-instructions per us, whole chip
    RUNTIME_SAC_PER_US = 15e6       # dense SACs per us on full tiles
    ROWS_SAC_PER_US = 9.6e6         # dense SACs per us, small-batch LinearShift kernel

    def estimate_us(self) -> float:
        """Modelled duration of one run of this plan on MI355X (see the cost
        model above)."""
        streams = max(1, self.segments * self.wsplit)
        executed = self.code_bytes / 4.2 * max(1, self.pixel_tiles) * max(1, self.pixel_groups)
        t = max(self.code_bytes / streams / self.PLAN_STREAM_BPUS, executed / self.PLAN_ISSUE_PER_US)
        est = 3.0 + (3.0 if self.splits > 1 else 0.0) + t
        return 2.5 + 1.16 * est if getattr(self, "transposed", False) else est

    def runtime_estimate_us(self) -> float:
        """Modelled duration of the same layer on the runtime kernel
        (ds_conv2d_shift / ds_linear_shift)."""
        nq = max(1, self.out_pixels)
        weight_bytes = self.out_channels * packed_row_words(self.crs) * 4
        if self.linear and nq < 256:
            return 5.5 + max(self.sac / self.ROWS_SAC_PER_US, weight_bytes / 1.75e6)
        fill = nq / (-(-nq // 256) * 256)
        return ((40.0 if self.linear else 25.0) + self.sac / (self.RUNTIME_SAC_PER_US * fill)
                + weight_bytes / 4e6)

    @property
    def preferred(self) -> bool:
        """Whether this plan is expected to beat the runtime kernel, by the cost
        model above. Measured on MI355X as graph replays (model in brackets),
        plan against runtime kernel: 4096 -> 4096 at batch 256 on x^T 104-109
        us (108) against 346 us (329); 2048 -> 1000 at batch 128 on x^T 17.0 us
        (17.5) against 32.5-36 us (33); 1024 -> 1024 at batch 64 on x^T 11.9 us
        (12.0) against 13.7 us (12.5); 512 -> 512 at batch 128 on x^T 10.3 us
        (12.0) against 8.4 us (9.0); 128 -> 128 3 x 3 at 28 x 28, batch 1 8.6 us
        (10) against 42 us eager (33); 256 -> 128 at batch 8 4.2 us (5.5)
        against 4.5 us (5.5); 512 -> 1000 at batch 32 10.2 us (11) against 6.5
        us (7.2); 25088 -> 4096 at batch 1 344 us (282) against 41 us (42). Over
        the layers of ResNet-18 (batch 32) and ResNet-50 (batch 128) measured /
        modelled plan durations have medians 1.16 and 1.04, runtime-kernel ones
        0.97 and 0.92."""
        return self.estimate_us() < self.runtime_estimate_us()

    def __call__(self, x: torch.Tensor, residual: torch.Tensor | None = None, out=None):
        _dev_int(x, "x", getattr(self, "act_bits", 32))
        if tuple(x.shape) != self.x_shape:
            raise ValueError(f"x must have shape {self.x_shape}")
        if residual is not None:
            _dev_i32(residual, "residual")
        y = out if out is not None else torch.empty(self.y_shape, dtype=torch.int32, device=x.device)
        _dev_i32(y, "out")
        args = (self._h, _ptr(x), _ptr(residual), _ptr(y), _stream(x.device))
        if x.device.index == torch.cuda.current_device():
            call("ds_jit_conv_run", *args)   # (entering the device context costs microseconds)
        else:
            with torch.cuda.device(x.device):
                call("ds_jit_conv_run", *args)
        return y

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().ds_jit_conv_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class JitConvBackwardData(JitConv):
    """A weight-specialised plan for the input gradient of a ConvShift layer
    (``ds_jit_conv_backward_data_create``): ``plan(dy)`` returns dx. The arguments
    describe the forward layer (x_shape = its input)."""

    def __init__(self, w_packed, x_shape, kernel_size, stride=1, padding=0, splits: int = 0,
                 device="cuda:0", code_bits: int = 5):
        self.k = int(w_packed.shape[0])
        wp, _, _, _ = _jit_args(w_packed, self.k, None, None, None)
        n, c, h, w = (int(v) for v in x_shape)
        r, s = _pair(kernel_size)
        sh, sw = _pair(stride)
        ph, pw = _pair(padding)
        self.x_shape = (n, self.k, out_size(h, ph, r, sh), out_size(w, pw, s, sw))   # dy
        self.y_shape = (n, c, h, w)                                                  # dx
        self.device = torch.device(device)
        self.residual = False
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            call("ds_jit_conv_backward_data_create", _np_ptr(wp), n, c, h, w, self.k, r, s, sh, sw,
                 ph, pw, code_bits_flag(code_bits), splits, ctypes.byref(handle))
        self._h = handle
        self._query()
        self.crs = self.k * r * s       # weights per input channel of the forward layer
        self.out_pixels, self.out_channels = n * h * w, c
        self.sac = n * self.k * self.x_shape[2] * self.x_shape[3] * c * r * s
        self.linear = False


def layer_plan(layer, w_packed, bias=None, device="cuda:0", act_bits: int = 32) -> JitConv:
    """The weight-specialised plan of one workload layer (an object with ``kind``
    "conv" or "linear", ``n, c, h, w, k, r, s, stride, pad``), made the way the
    benchmark makes it: a LinearShift [batch, in] -> [batch, out] is the 1 x 1
    ConvShift of [batch, in, 1, 1]. ``w_packed``: host packed codes [k, words]."""
    if layer.kind == "linear":
        return JitConv(w_packed, (layer.n, layer.c, 1, 1), 1, 1, 0, bias=bias, device=device,
                       act_bits=act_bits)
    return JitConv(w_packed, (layer.n, layer.c, layer.h, layer.w), (layer.r, layer.s), layer.stride,
                   layer.pad, bias=bias, device=device, act_bits=act_bits)


def run_layer_plan(plan: JitConv, layer, x: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """Runs a plan of ``layer_plan`` on the layer's own input layout ([batch, in] for a
    LinearShift) and returns y in the layer's output layout."""
    if layer.kind == "linear":
        y4 = plan(x.view(layer.n, layer.c, 1, 1), out=None if out is None else out.view(layer.n, layer.k, 1, 1))
        return y4.view(layer.n, layer.k)
    return plan(x, out=out)


def set_tuning(name: str, value: int) -> None:
    """Sets a tuning override of the library (``ds_set_tuning``): "DS_FORCE_VARIANT",
    "DS_JIT_WSPLIT", "DS_JIT_SLOTS", "DS_JIT_MAP", "DS_JIT_GROUP_TILES",
    "DS_JIT_ORDER", "DS_JIT_TN", "DS_JIT_PGROUPS", "DS_JIT_TRANSPOSE" or
    "DS_ROWS_BATCH"; a negative value restores the library's own choice."""
    call("ds_set_tuning", name.encode(), int(value))


def get_tuning(name: str) -> int:
    v = ctypes.c_int32()
    call("ds_get_tuning", name.encode(), ctypes.byref(v))
    return v.value


class tuning:
    """Context manager: ``with ops.tuning("DS_FORCE_VARIANT", 0): ...`` sets a tuning
    override for the block and restores the previous value afterwards."""

    def __init__(self, name: str, value: int):
        self.name, self.value = name, value

    def __enter__(self):
        self.prev = get_tuning(self.name)
        set_tuning(self.name, self.value)
        return self

    def __exit__(self, *exc):
        set_tuning(self.name, self.prev)
        return False


def _mul_weights(w, k):
    a = np.ascontiguousarray(w.cpu().numpy() if isinstance(w, torch.Tensor) else w)
    if a.dtype != np.int32 or a.ndim != 2 or a.shape[0] != k:
        raise ValueError("w must be int32 [k, c*r*s]")
    return a


def jit_conv_mul_image(w, x_shape, kernel_size, stride=1, padding=0, bias=None, relu: bool = False,
                       splits: int = 0) -> bytes:
    """The code object a JitConvMul with these arguments would load (host only)."""
    k = int(w.shape[0])
    wa, b = _mul_weights(w, k), _host_i32(bias, k, "bias")
    n, c, h, wd = x_shape
    r, s = _pair(kernel_size)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    size = ctypes.c_int64(0)
    args = [_np_ptr(wa), _np_ptr(b), n, c, h, wd, k, r, s, sh, sw, ph, pw, DS_RELU if relu else 0, splits]
    st = lib().ds_jit_conv_mul_image(*args, None, 0, ctypes.byref(size))
    if st not in (0, 4):
        call("ds_jit_conv_mul_image", *args, None, 0, ctypes.byref(size))
    buf = ctypes.create_string_buffer(size.value)
    call("ds_jit_conv_mul_image", *args, buf, size.value, ctypes.byref(size))
    return buf.raw[:size.value]


class JitConvMul(JitConv):
    """A multiplication plan (``ds_jit_conv_mul_create``): the comparison operator
    y = bias + sum x * w (24-bit signed operands) in the shift plans' tiling, with
    int32 weights w [k, c*r*s] baked into the code."""

    def __init__(self, w, x_shape, kernel_size, stride=1, padding=0, bias=None, relu: bool = False,
                 splits: int = 0, device="cuda:0"):
        self.k = int(w.shape[0])
        wa, b = _mul_weights(w, self.k), _host_i32(bias, self.k, "bias")
        self.x_shape = tuple(int(v) for v in x_shape)
        n, c, h, wd = self.x_shape
        r, s = _pair(kernel_size)
        sh, sw = _pair(stride)
        ph, pw = _pair(padding)
        self.y_shape = (n, self.k, out_size(h, ph, r, sh), out_size(wd, pw, s, sw))
        self.device = torch.device(device)
        self.residual = False
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            call("ds_jit_conv_mul_create", _np_ptr(wa), _np_ptr(b), n, c, h, wd, self.k, r, s, sh, sw,
                 ph, pw, DS_RELU if relu else 0, splits, ctypes.byref(handle))
        self._h = handle
        self._query()
        self.crs = c * r * s
        self.out_pixels, self.out_channels = n * self.y_shape[2] * self.y_shape[3], self.k
        self.sac = self.out_pixels * self.k * self.crs
        self.linear = h == wd == r == s == 1 and ph == pw == 0
