"""C-ABI checks that need no GPU: symbols, packing, and argument validation.

Validation runs before any device access, so NULL pointers, bad shapes and
bad arguments are rejected here with the documented status and nothing is
written. Compute calls themselves need a GPU and live in the gpu suite.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_1905_13298_amd import _native, ops
from paper_1905_13298_amd.workloads import random_codes

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "deepshift.h")

OK, NULLP, SHAPE, ARG, SMALL, CODE, HIP, UNSUP = range(8)
FAKE = 0x10000  # never dereferenced: every case below fails validation first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ds_\w+)\s*\(", text)))


def test_header_symbols_exported():
    names = declared_functions()
    assert len(names) >= 9
    lib = ctypes.CDLL(_native.library_path())
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(_native.SIGNATURES)


def test_status_strings():
    lib = _native.lib()
    seen = set()
    for st in range(8):
        s = lib.ds_status_string(st).decode()
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 8
    assert lib.ds_status_string(99).decode() == "unknown status"


def test_packed_row_words():
    lib = _native.lib()
    for cols, words in [(1, 1), (6, 1), (7, 2), (12, 2), (13, 3), (147, 25), (4096, 683)]:
        assert lib.ds_packed_row_words(cols) == words
    assert lib.ds_packed_row_words(0) == -1 and lib.ds_packed_row_words(-5) == -1


@pytest.mark.parametrize("cols", [1, 5, 6, 7, 13, 64, 147, 576, 1152, 4096])
def test_pack_matches_oracle_layout(cols):
    rng = np.random.default_rng(cols)
    codes = rng.integers(0, 32, (5, cols)).astype(np.uint8)
    got = ops.pack_shift_weights(codes)
    np.testing.assert_array_equal(got, oracle.pack_codes(codes))
    np.testing.assert_array_equal(ops.unpack_shift_weights(got, cols), codes)


def test_pack_errors_write_nothing():
    lib = _native.lib()
    codes = np.zeros((2, 7), np.uint8)
    out = np.full(4, 0xDEADBEEF, np.uint32)
    p, o = codes.ctypes.data, out.ctypes.data
    assert lib.ds_pack_shift_weights(None, 2, 7, o, 4) == NULLP
    assert lib.ds_pack_shift_weights(p, 2, 7, None, 4) == NULLP
    assert lib.ds_pack_shift_weights(p, 0, 7, o, 4) == SHAPE
    assert lib.ds_pack_shift_weights(p, 2, -1, o, 4) == SHAPE
    assert lib.ds_pack_shift_weights(p, 2, 7, o, 3) == SMALL
    codes[1, 6] = 32
    assert lib.ds_pack_shift_weights(p, 2, 7, o, 4) == CODE
    assert "32" in lib.ds_last_error_message().decode()
    assert np.all(out == 0xDEADBEEF)
    codes[1, 6] = 31
    assert lib.ds_pack_shift_weights(p, 2, 7, o, 4) == OK
    assert lib.ds_last_error_message().decode() == ""


def test_unpack_errors():
    lib = _native.lib()
    words = np.array([[0x0C520C41]], np.uint32)
    out = np.full(6, 0xAA, np.uint8)
    assert lib.ds_unpack_shift_weights(words.ctypes.data, 1, 6, out.ctypes.data, 5) == SMALL
    bad = np.array([[1 << 30]], np.uint32)
    assert lib.ds_unpack_shift_weights(bad.ctypes.data, 1, 6, out.ctypes.data, 6) == CODE
    assert np.all(out == 0xAA)
    assert lib.ds_unpack_shift_weights(words.ctypes.data, 1, 6, out.ctypes.data, 6) == OK
    np.testing.assert_array_equal(out, [1, 2, 3, 4, 5, 6])


def conv(**kw):
    a = dict(x=FAKE, w=FAKE + 4096, b=None, y=FAKE + 8192, n=1, c=2, h=5, wd=5, k=3, r=3, s=3,
             sh=1, sw=1, ph=1, pw=1, f=16, flags=0)
    a.update(kw)
    return _native.lib().ds_conv2d_shift(a["x"], a["w"], a["b"], a["y"], a["n"], a["c"], a["h"],
                                          a["wd"], a["k"], a["r"], a["s"], a["sh"], a["sw"],
                                          a["ph"], a["pw"], a["f"], a["flags"], None)


def test_conv_validation_codes():
    assert conv(x=None) == NULLP
    assert conv(w=None) == NULLP
    assert conv(y=None) == NULLP
    for key in ("n", "c", "h", "wd", "k", "r", "s"):
        assert conv(**{key: 0}) == SHAPE, key
        assert conv(**{key: -2}) == SHAPE, key
    assert conv(r=9, ph=1) == SHAPE           # kernel larger than padded input
    assert conv(sh=0) == ARG and conv(sw=-1) == ARG
    assert conv(ph=-1) == ARG
    assert conv(f=-1) == ARG and conv(f=32) == ARG
    assert conv(flags=2) == ARG and conv(flags=0x80000000) == ARG
    assert conv(n=1 << 20, c=1 << 12, h=1, wd=1) == UNSUP
    assert conv(k=1 << 17, c=1 << 14, r=1, s=1, ph=0, pw=0) == UNSUP
    # y overlapping x
    assert conv(y=FAKE + 4) == ARG
    assert "overlap" in _native.lib().ds_last_error_message().decode()


def test_linear_and_mul_validation_codes():
    lib = _native.lib()
    assert lib.ds_linear_shift(None, FAKE, None, FAKE * 4, 2, 3, 4, 16, 0, None) == NULLP
    assert lib.ds_linear_shift(FAKE, FAKE * 2, None, FAKE * 4, 0, 3, 4, 16, 0, None) == SHAPE
    assert lib.ds_linear_shift(FAKE, FAKE * 2, None, FAKE * 4, 2, 3, 4, 40, 0, None) == ARG
    assert lib.ds_linear_shift(FAKE, FAKE * 2, None, FAKE * 4, 2, 3, 4, 16, 2, None) == ARG
    assert lib.ds_linear_mul_i32(FAKE, None, None, FAKE * 4, 2, 3, 4, 0, None) == NULLP
    assert lib.ds_conv2d_mul_i32(FAKE, FAKE * 2, None, FAKE * 4, 1, 1, 4, 4, 1, 3, 3,
                                 0, 1, 0, 0, 0, None) == ARG


def test_host_pointers_rejected_without_gpu_access():
    """Host memory is not a device buffer: DS_ERR_INVALID_ARG (HIP lookup fails)."""
    x = np.zeros((2, 4), np.int32)
    w = ops.pack_shift_weights(random_codes(np.random.default_rng(0), (3, 4)))
    y = np.full((2, 3), 7, np.int32)
    st = _native.lib().ds_linear_shift(x.ctypes.data, w.ctypes.data, None, y.ctypes.data,
                                        2, 4, 3, 16, 0, None)
    assert st in (ARG, HIP)
    assert np.all(y == 7)


def test_describe_names_a_kernel_without_a_gpu():
    assert ops.describe_conv2d(128, 64, 56, 56, 256, 1).startswith("tiled point")
    assert ops.describe_conv2d(128, 64, 56, 56, 64, 3, 1, 1).startswith("tiled window")
    assert ops.describe_conv2d(2, 3, 224, 224, 64, 7, 2, 3).startswith("tiled window")
    assert ops.describe_conv2d(1, 3, 9, 9, 5, 4, 1, 1).startswith("tiled window tm4 cc1 s4")
    assert ops.describe_conv2d(1, 3, 12, 12, 5, 6, 1, 1) == "direct"   # no instance for 6 taps per row
    # LinearShift (1 x 1 on 1 x 1 inputs) below 256 rows: the small-batch kernel
    assert ops.describe_conv2d(1, 25088, 1, 1, 4096, 1) == "rows"
    assert ops.describe_conv2d(255, 2048, 1, 1, 1000, 1) == "rows"
    assert ops.describe_conv2d(256, 4096, 1, 1, 4096, 1).startswith("tiled point transposed")
    assert ops.describe_conv2d(8, 256, 2, 1, 128, 1).startswith("tiled")
    lib = _native.lib()
    import ctypes
    buf = ctypes.create_string_buffer(4)
    assert lib.ds_conv2d_shift_describe(1, 1, 1, 1, 1, 1, 1, 1, 1, 0, 0, buf, 4) == OK
    assert len(buf.value) <= 3
    assert lib.ds_conv2d_shift_describe(0, 1, 1, 1, 1, 1, 1, 1, 1, 0, 0, buf, 4) == SHAPE
    assert lib.ds_conv2d_shift_describe(1, 1, 1, 1, 1, 1, 1, 1, 1, 0, 0, None, 4) == NULLP


def test_converter_validation_codes():
    lib = _native.lib()
    q, ps, fx = lib.ds_quantize_shift_weights_q, lib.ds_quantize_shift_weights_ps, lib.ds_to_fixed_point
    assert q(None, 2, 6, 14, FAKE * 4, 0, None) == NULLP
    assert q(FAKE, 2, 6, 14, None, 0, None) == NULLP
    assert q(FAKE, 0, 6, 14, FAKE * 4, 0, None) == SHAPE
    assert q(FAKE, 2, -1, 14, FAKE * 4, 0, None) == SHAPE
    assert q(FAKE, 2, 6, 15, FAKE * 4, 0, None) == ARG
    assert q(FAKE, 2, 6, -1, FAKE * 4, 0, None) == ARG
    assert q(FAKE, 2, 6, 14, FAKE * 4, 1, None) == ARG
    assert q(FAKE, 2, 6, 14, FAKE * 4, 3 << 8, None) == ARG    # shifts to -14 need 5 bits
    assert "does not fit" in lib.ds_last_error_message().decode()
    assert q(FAKE, 2, 6, 2, FAKE * 4, 7 << 8, None) == ARG     # no 7-bit codes
    assert q(FAKE, 1 << 16, 1 << 15, 14, FAKE * 4, 0, None) == UNSUP
    assert q(FAKE, 2, 6, 14, FAKE + 8, 0, None) == ARG     # output overlaps w
    assert "overlap" in lib.ds_last_error_message().decode()
    assert ps(FAKE, None, 2, 6, 14, FAKE * 4, 0, None) == NULLP
    assert ps(FAKE, FAKE * 2, 2, 6, 14, FAKE * 2 + 4, 0, None) == ARG   # overlaps s
    assert ps(FAKE, FAKE * 2, 2, 0, 14, FAKE * 4, 0, None) == SHAPE
    assert fx(None, 4, 16, FAKE * 4, 0, None) == NULLP
    assert fx(FAKE, 0, 16, FAKE * 4, 0, None) == SHAPE
    assert fx(FAKE, 4, 32, FAKE * 4, 0, None) == ARG
    assert fx(FAKE, 4, -1, FAKE * 4, 0, None) == ARG
    assert fx(FAKE, 4, 16, FAKE * 4, 3, None) == ARG
    assert fx(FAKE, 1 << 31, 16, FAKE * 4, 0, None) == UNSUP
    assert fx(FAKE, 4, 16, FAKE + 4, 0, None) == ARG       # partial overlap


def test_converter_rejects_host_buffers():
    lib = _native.lib()
    w = np.ones((2, 6), np.float32)
    out = np.full((2, 1), 7, np.uint32)
    assert lib.ds_quantize_shift_weights_q(w.ctypes.data, 2, 6, 14, out.ctypes.data, 0, None) in (ARG, HIP)
    y = np.full(12, 7, np.int32)
    assert lib.ds_to_fixed_point(w.ctypes.data, 12, 16, y.ctypes.data, 0, None) in (ARG, HIP)
    assert np.all(out == 7) and np.all(y == 7)


def test_converter_many_validation_codes():
    lib = _native.lib()
    many = lib.ds_quantize_shift_weights_q_many
    P2 = ctypes.c_void_p * 2
    I2 = ctypes.c_int64 * 2
    w = P2(FAKE, FAKE * 2)
    out = P2(FAKE * 4, FAKE * 8)
    assert many(0, w, I2(2, 2), I2(6, 6), 14, out, 0, None) == SHAPE
    assert many(2, None, I2(2, 2), I2(6, 6), 14, out, 0, None) == NULLP
    assert many(2, w, None, I2(6, 6), 14, out, 0, None) == NULLP
    assert many(2, w, I2(2, 0), I2(6, 6), 14, out, 0, None) == SHAPE
    assert "tensor 1" in lib.ds_last_error_message().decode()
    assert many(2, P2(FAKE, None), I2(2, 2), I2(6, 6), 14, out, 0, None) == NULLP
    assert many(2, w, I2(2, 2), I2(6, 6), 15, out, 0, None) == ARG
    # two outputs on top of each other
    assert many(2, w, I2(2, 2), I2(6, 6), 14, P2(FAKE * 4, FAKE * 4), 0, None) in (ARG,)


def test_fused_and_pool_validation_codes():
    lib = _native.lib()
    fused = lib.ds_conv2d_shift_fused

    def fz(**kw):
        a = dict(x=FAKE, w=FAKE + 4096, b=None, mul=FAKE + 6000, add=None, ms=16, res=None,
                 y=FAKE + 8192, flags=0)
        a.update(kw)
        return fused(a["x"], a["w"], a["b"], a["mul"], a["add"], a["ms"], a["res"], a["y"],
                     1, 2, 5, 5, 3, 3, 3, 1, 1, 1, 1, 16, a["flags"], None)
    assert fz(x=None) == NULLP
    assert fz(flags=2) == ARG
    assert fz(mul=None, add=FAKE + 7000) == ARG
    assert "add needs mul" in lib.ds_last_error_message().decode()
    assert fz(ms=32) == ARG and fz(ms=-1) == ARG
    assert fz(res=FAKE + 8192 + 8) == ARG          # residual overlapping y
    assert "overlap" in lib.ds_last_error_message().decode()
    mp = lib.ds_maxpool2d
    assert mp(None, FAKE, 1, 1, 8, 8, 3, 3, 2, 2, 1, 1, 0, None) == NULLP
    assert mp(FAKE, FAKE * 4, 0, 1, 8, 8, 3, 3, 2, 2, 1, 1, 0, None) == SHAPE
    assert mp(FAKE, FAKE * 4, 1, 1, 8, 8, 3, 3, 2, 2, 2, 1, 0, None) == ARG   # pad > r/2
    assert mp(FAKE, FAKE * 4, 1, 1, 8, 8, 3, 3, 0, 2, 1, 1, 0, None) == ARG   # stride 0
    assert mp(FAKE, FAKE * 4, 1, 1, 8, 8, 3, 3, 2, 2, 1, 1, 1, None) == ARG   # flags
    assert mp(FAKE, FAKE + 4, 1, 1, 8, 8, 3, 3, 2, 2, 1, 1, 0, None) == ARG   # overlap
    ap = lib.ds_avgpool2d_global
    assert ap(FAKE, None, 1, 1, 7, 7, 0, None) == NULLP
    assert ap(FAKE, FAKE * 4, 1, 0, 7, 7, 0, None) == SHAPE
    assert ap(FAKE, FAKE * 4, 1, 1, 7, 7, 4, None) == ARG


def test_backward_validation_codes():
    lib = _native.lib()
    a = [FAKE, FAKE * 2, FAKE * 4, 1, 2, 6, 6, 3, 3, 3, 1, 1, 1, 1, 16, 0, None]

    def bwd(**kw):
        v = list(a)
        keys = ["dy", "w", "dx", "n", "c", "h", "wd", "k", "r", "s", "sh", "sw", "ph", "pw", "f", "flags"]
        for key, val in kw.items():
            v[keys.index(key)] = val
        return lib.ds_conv2d_shift_backward_data(*v)

    assert bwd(dy=None) == NULLP and bwd(w=None) == NULLP and bwd(dx=None) == NULLP
    for key in ("n", "c", "h", "wd", "k", "r", "s"):
        assert bwd(**{key: 0}) == SHAPE, key
    assert bwd(r=9) == SHAPE
    assert bwd(sh=0) == ARG and bwd(pw=-1) == ARG
    assert bwd(f=32) == ARG and bwd(flags=1) == ARG
    assert bwd(n=1 << 20, c=1 << 12, h=1, wd=1, r=1, s=1, ph=0, pw=0) == UNSUP
    assert bwd(dx=FAKE + 4) == ARG                       # dx overlapping dy
    assert "overlap" in lib.ds_last_error_message().decode()
    assert lib.ds_linear_shift_backward_data(None, FAKE, FAKE * 4, 2, 3, 4, 16, 0, None) == NULLP
    assert lib.ds_linear_shift_backward_data(FAKE, FAKE * 2, FAKE * 4, 0, 3, 4, 16, 0, None) == SHAPE
    assert lib.ds_linear_shift_backward_data(FAKE, FAKE * 2, FAKE * 4, 2, 3, 4, 16, 4, None) == ARG
    # host buffers are not device buffers; nothing is written
    dy = np.zeros((2, 4), np.int32)
    w = ops.pack_shift_weights(random_codes(np.random.default_rng(0), (4, 3)))
    dx = np.full((2, 3), 7, np.int32)
    st = lib.ds_linear_shift_backward_data(dy.ctypes.data, w.ctypes.data, dx.ctypes.data, 2, 3, 4,
                                           16, 0, None)
    assert st in (ARG, HIP) and np.all(dx == 7)


def test_backward_describe_plans_phases_without_a_gpu():
    d = ops.describe_conv2d_backward_data
    s2 = d(128, 64, 56, 56, 128, 3, 2, 1)
    assert s2.startswith("phases4") and s2.count("tiled") == 4
    assert d(128, 64, 56, 56, 64, 3, 1, 1).startswith("phases1; 3x3 tiled window")
    ds = d(128, 1024, 14, 14, 2048, 1, 2, 0)
    assert ds.startswith("phases4; 1x1 tiled point") and ds.count("zero") == 3
    assert d(256, 4096, 1, 1, 4096, 1).startswith("phases1; 1x1 tiled point transposed")
    stem = d(2, 3, 224, 224, 64, 7, 2, 3)                       # phases of 3 and 4 taps per row
    assert stem.startswith("phases4") and stem.count("tiled") == 4 and stem.count(" s4 ") == 2
    assert d(1, 3, 6, 6, 2, 1, 1, 1) == "direct"               # padding beyond the window
    with pytest.raises(ops.DeepShiftError, match="INVALID_SHAPE"):
        d(1, 1, 2, 2, 1, 3, 1, 0)


def test_tuning_overrides_are_explicit():
    """Tuning knobs start from the environment at load and change only through
    ds_set_tuning; unknown names and NULL pointers are rejected."""
    from paper_1905_13298_amd import ops
    lib = _native.lib()
    before = ops.get_tuning("DS_JIT_ORDER")
    try:
        ops.set_tuning("DS_JIT_ORDER", 2)
        assert ops.get_tuning("DS_JIT_ORDER") == 2
        with ops.tuning("DS_JIT_ORDER", 1):
            assert ops.get_tuning("DS_JIT_ORDER") == 1
        assert ops.get_tuning("DS_JIT_ORDER") == 2
        ops.set_tuning("DS_JIT_ORDER", -7)
        assert ops.get_tuning("DS_JIT_ORDER") == -1
    finally:
        ops.set_tuning("DS_JIT_ORDER", before)
    for name in ("DS_FORCE_VARIANT", "DS_JIT_WSPLIT", "DS_JIT_SLOTS", "DS_JIT_MAP", "DS_JIT_GROUP_TILES",
                 "DS_JIT_ORDER", "DS_JIT_TN", "DS_JIT_PGROUPS", "DS_JIT_TRANSPOSE", "DS_ROWS_BATCH"):
        ops.get_tuning(name)   # every documented knob is known
    assert lib.ds_set_tuning(b"DS_NO_SUCH_KNOB", 1) == 3
    assert lib.ds_set_tuning(None, 1) == 1
    assert lib.ds_get_tuning(b"DS_JIT_SLOTS", None) == 1
    # The environment is not read again after load.
    import os
    loaded = ops.get_tuning("DS_JIT_WSPLIT")
    old = os.environ.get("DS_JIT_WSPLIT")
    os.environ["DS_JIT_WSPLIT"] = "4" if loaded != 4 else "2"
    try:
        assert ops.get_tuning("DS_JIT_WSPLIT") == loaded
    finally:
        if old is None:
            del os.environ["DS_JIT_WSPLIT"]
        else:
            os.environ["DS_JIT_WSPLIT"] = old


def test_noalloc_limit_checked_from_the_shape_alone():
    """ds_conv2d_shift_noalloc rejects a problem whose scratch exceeds its array
    before touching any buffer; the scratch query needs no GPU."""
    lib = _native.lib()
    need = lib.ds_conv2d_shift_noalloc_scratch_bytes(256, 4096, 1, 1, 4096, 1, 1, 1, 1, 0, 0)
    assert need > (32 << 20)
    assert lib.ds_conv2d_shift_noalloc_scratch_bytes(1, 128, 28, 28, 128, 3, 3, 1, 1, 1, 1) <= (32 << 20)
    assert lib.ds_conv2d_shift_noalloc_scratch_bytes(0, 1, 1, 1, 1, 1, 1, 1, 1, 0, 0) == -1
    # the small-batch LinearShift kernel needs no scratch at any size
    assert lib.ds_conv2d_shift_noalloc_scratch_bytes(255, 25088, 1, 1, 4096, 1, 1, 1, 1, 0, 0) == 0
    x = np.zeros(16, np.int32)
    st = lib.ds_conv2d_shift_noalloc(x.ctypes.data, x.ctypes.data, None, x.ctypes.data, 256, 4096, 1,
                                     1, 4096, 1, 1, 1, 1, 0, 0, 16, 0, None)
    assert st == 7 and b"scratch" in lib.ds_last_error_message()
    # Within the limit, host buffers are rejected as for ds_conv2d_shift.
    st = lib.ds_conv2d_shift_noalloc(x.ctypes.data, x.ctypes.data, None, x.ctypes.data, 1, 2, 2, 2,
                                     2, 1, 1, 1, 1, 0, 0, 16, 0, None)
    assert st == 3
