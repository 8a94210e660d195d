"""CPU checks of the weight-specialised ConvShift code generator.

``ds_jit_conv_image`` returns the code object a plan would load; no GPU is
needed. The tests

* check the ELF structure: the generated code is the last loadable segment and
  lies past every other one;
* disassemble it with llvm-objdump (an encoder mistake shows up as an unknown or
  different instruction) and run it in a small interpreter of the dozen gfx950
  instructions the generator emits, over every lane of every pixel tile at
  once. The lane inputs (tap and output offsets) follow the template kernel's
  index arithmetic. The interpreter checks that every in-range buffer access
  stays inside its buffer (with the range check taken either with or without
  the scalar offset), that no register is read before the s_waitcnt that
  covers its load, and that each lane stores each output once. The result is
  compared with the oracle's convolution and epilogue.
"""
import collections
import zlib
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_1905_13298_amd import ops

LLVM = "/opt/rocm/llvm/bin"
OOB = 0x80000000
M32 = 0xFFFFFFFF


def gen_layer(seed, n, c, h, w, k, r, s, zero_frac=0.1):
    rng = np.random.default_rng(seed)
    sign = rng.integers(0, 2, (k, c * r * s))
    shift = rng.integers(0, 15, (k, c * r * s))
    shift[rng.random(shift.shape) < zero_frac] = 15
    codes = (sign << 4 | shift).astype(np.uint8)
    x = rng.integers(-(2 ** 31), 2 ** 31, (n, c, h, w), dtype=np.int64).astype(np.int32)
    return codes, x, rng


def disassemble(img, tmp_path):
    path = os.path.join(tmp_path, "plan.hsaco")
    with open(path, "wb") as f:
        f.write(img)
    out = subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", path], capture_output=True,
                         text=True, check=True).stdout
    insts, body = {}, False
    for line in out.splitlines():
        if line.startswith("Disassembly of section"):
            body = ".jitbody" in line
            continue
        if not body or "//" not in line:
            continue
        code, comment = line.split("//", 1)
        addr, words = comment.strip().split(":", 1)
        parts = code.replace(",", " ").split()
        insts[int(addr, 16)] = (parts[0], parts[1:], int(addr, 16) + 4 * len(words.split()))
    return insts


def elf_layout(img):
    rd = subprocess.run([f"{LLVM}/llvm-readelf", "-lS", "-W", "/dev/stdin"], input=img,
                        capture_output=True, check=True).stdout.decode()
    loads = [ln.split() for ln in rd.splitlines() if ln.strip().startswith("LOAD")]
    sec = [ln for ln in rd.splitlines() if ".jitbody" in ln and "PROGBITS" in ln][0].split()
    i = sec.index("PROGBITS")
    return loads, int(sec[i + 1], 16), int(sec[i + 2], 16), int(sec[i + 3], 16)


def padded_extents(h, w, r, s, st, pd):
    """Windows over 3 x 3 read a zero-padded copy of x with the extents the
    windows reach; None for smaller windows."""
    if r <= 3 and s <= 3:
        return None
    oh, ow = (h + 2 * pd - r) // st + 1, (w + 2 * pd - s) // st + 1
    return (oh - 1) * st + r, (ow - 1) * st + s


def pad_input(x, pd, xh, xw):
    n, c, h, w = x.shape
    xp = np.zeros((n, c, xh + h + pd, xw + w + pd), x.dtype)
    xp[:, :, pd:pd + h, pd:pd + w] = x
    return xp[:, :, :xh, :xw]


def default_pgroups(wsplit):
    return 4 // wsplit if wsplit <= 4 else 1


def lane_inputs(n, c, h, w, k, r, s, st, pd, wsplit=1, pgroups=None):
    """Per lane (pixel q of every 256-pixel tile): tap byte offsets v4..v12 of
    the 3 x 3 window at channel 0 and the output byte offset v13, as the
    template kernel computes them (past-the-end marker for padding and for
    lanes beyond the last pixel). For a window over 3 x 3 the template sees
    the padded copy of x as an unpadded input."""
    oh, ow = (h + 2 * pd - r) // st + 1, (w + 2 * pd - s) // st + 1
    ext = padded_extents(h, w, r, s, st, pd)
    if ext is not None:
        h, w, pd = ext[0], ext[1], 0
    nq = n * oh * ow
    lanes = -(-nq // 256) * 256
    q = np.arange(lanes)
    valid = q < nq
    nn, pix = q // (oh * ow), q % (oh * ow)
    ohh, oww = pix // ow, pix % ow
    regs = {}
    for rr in range(3):
        for ss in range(3):
            ih, iw = ohh * st - pd + rr, oww * st - pd + ss
            ok = valid & (ih >= 0) & (ih < h) & (iw >= 0) & (iw < w)
            regs[4 + rr * 3 + ss] = np.where(ok, (nn * c * h * w + ih * w + iw) * 4, OOB).astype(np.int64)
    regs[13] = np.where(valid, (nn * k * oh * ow + pix) * 4, OOB).astype(np.int64)
    # v3: LDS byte offset of the lane's pixel in its workgroup (wave split; a
    # workgroup covers 64 pixels per pixel group)
    within = q % (64 * (pgroups or default_pgroups(wsplit)))
    regs[3] = ((within // 64) * 16384 + (within % 64) * 4).astype(np.int64)
    return regs, (oh, ow)


def transposed_linear(n, h, w, r, s):
    """A LinearShift plan of batch >= 32 (>= 2 with DS_JIT_TRANSPOSE = 1, none with
    0) runs its kernel on x^T [c][n] (an int32 copy the plan makes) as one image of
    1 x n pixels, writing y^T [k][n]; a last pass transposes y^T into y, adding the
    residual and applying the ReLU of a layer with a residual (the kernel then
    applies neither)."""
    forced = ops.get_tuning("DS_JIT_TRANSPOSE")
    least = {0: 1 << 62, 1: 2}.get(forced, 32)
    return h == w == r == s == 1 and n >= least


def plan_lanes(n, c, h, w, k, r, s, st, pd, wsplit=1, pgroups=None):
    """lane_inputs for the problem the plan's kernel sees (see transposed_linear)."""
    if not transposed_linear(n, h, w, r, s):
        return lane_inputs(n, c, h, w, k, r, s, st, pd, wsplit, pgroups)
    lanes, _ = lane_inputs(1, c, 1, n, k, 1, 1, 1, 0, wsplit, pgroups)
    return lanes, (1, 1)


def y_start(bias, n, k, oh, ow, transposed):
    """y (or y^T) as the split-K fill pass leaves it: the bias of each channel."""
    b = bias.view(np.uint32).astype(np.int64)
    return np.repeat(b, n) if transposed else np.repeat(np.tile(b, n), oh * ow)


def transpose_back(y, n, k, res=None, relu=False):
    """The last pass of a transposed LinearShift: y^T [k][n] -> y [n][k], plus the
    residual, then the ReLU when there is a residual."""
    out = to_i32(y).reshape(k, n).T.astype(np.int64)
    if res is not None:
        out = out + res.reshape(n, k).astype(np.int64)
        if relu:
            out = np.maximum(to_i32(out), 0)
    return np.ascontiguousarray(out).reshape(-1).astype(np.int64) & M32


def x_buffer(x, r, s, st, pd):
    """The buffer the kernel reads x from (uint32 words as int64) and its bytes:
    x itself, its zero-padded copy (windows over 3 x 3) or its transposed copy."""
    n, c, h, w = x.shape
    if transposed_linear(n, h, w, r, s):
        xr = np.ascontiguousarray(x.reshape(n, c).T.astype(np.int32))
    else:
        ext = padded_extents(h, w, r, s, st, pd)
        xr = x if ext is None else pad_input(x, pd, *ext)
    xb = np.ascontiguousarray(xr).reshape(-1).view(np.uint32).astype(np.int64)
    return xb, xb.size * 4


class Interp:
    """The generated code, run for all lanes of one segment. ``run`` is a
    generator that stops at each s_barrier, so that the waves sharing pixels
    (wave split) can be run up to the barrier one after the other. LDS is one
    row of 64 channels per lane (pixel); an LDS access must land in the lane's
    own row."""

    def __init__(self, insts, bufs, wsplit=1, pgroups=None):
        self.insts, self.bufs = insts, bufs   # bufs: sgpr base -> (uint32 array, num_records)
        self.wsplit = wsplit
        self.pgroups = pgroups or default_pgroups(wsplit)

    @staticmethod
    def reg(tok):
        m = re.fullmatch(r"([vs])(\d+)", tok)
        return (m.group(1), int(m.group(2))) if m else None

    def run(self, start, seg, lanes, y, atomic_ok, lds, stored):
        V = {i: a.copy() for i, a in lanes.items()}
        S = {19: seg}
        pending = collections.OrderedDict()   # vgpr -> value, in issue order
        lgkm = {}                              # vgpr -> value of an LDS read in flight
        q = np.arange(V[3].size)
        tile_px = 64 * self.pgroups
        pc = start
        steps = 0

        def val(tok):
            rg = self.reg(tok)
            if rg is None:
                return int(tok, 0) & M32
            kind, i = rg
            if kind == "s":
                return S[i] & M32
            assert i not in pending and i not in lgkm, f"v{i} read before its load completed (pc {pc:#x})"
            return V[i]

        def lds_row(ops_, imm_tok):
            off = V[int(ops_[0][1:])] + int(imm_tok.split(":")[1]) if imm_tok else V[int(ops_[0][1:])]
            j, rem = (off % 16384) // 256, off % 256
            assert np.all((off // 16384) * 64 + rem // 4 == q % tile_px), "LDS access outside the lane's row"
            assert np.all(j == j[0]) and 0 <= j[0] < 64
            return int(j[0])

        def sq(tok):
            return int(re.fullmatch(r"s\[(\d+):\d+\]", tok).group(1))

        def access(ops, size=4):
            base = sq(ops[2])
            arr, nrec = self.bufs[base]
            voff = V[int(ops[1][1:])].astype(np.int64)
            soff = S[int(ops[3][1:])] & M32
            imm = [int(t.split(":")[1]) for t in ops[4:] if t.startswith("offset:")]
            tot = voff + soff + (imm[0] if imm else 0)
            inr = voff < nrec
            assert not np.any(inr & (tot + size > nrec)), f"out-of-range access at pc {pc:#x}"
            assert not np.any(inr & (tot % size != 0))
            return arr, inr, tot // size

        while True:
            steps += 1
            assert steps < 50_000_000
            op, ops, nxt = self.insts[pc]
            if op == "s_getpc_b64":
                S[28], S[29] = nxt & M32, nxt >> 32
            elif op in ("s_add_u32", "s_addc_u32"):
                d = int(ops[0][1:])
                t = val(ops[1]) + val(ops[2]) + (S.get("scc", 0) if op == "s_addc_u32" else 0)
                S[d], S["scc"] = t & M32, t >> 32
            elif op == "s_setpc_b64":
                nxt = S[28] | (S[29] << 32)
            elif op == "s_mov_b32":
                S[int(ops[0][1:])] = val(ops[1])
            elif op == "s_waitcnt":
                m = re.fullmatch(r"vmcnt\((\d+)\)", ops[0])
                if m:
                    keep = int(m.group(1))
                    while len(pending) > keep:
                        i, v = pending.popitem(last=False)
                        V[i] = v
                else:
                    assert ops[0] == "lgkmcnt(0)", ops
                    V.update(lgkm)
                    lgkm.clear()
            elif op == "s_barrier":
                assert not lgkm and not pending
                yield pc
            elif op == "ds_add_u32":
                j = lds_row(ops[:1], next((t for t in ops[2:] if t.startswith("offset:")), None))
                lds[:, j] = (lds[:, j] + val(ops[1])) & M32
            elif op == "ds_read_b32":
                j = lds_row(ops[1:2], next((t for t in ops[2:] if t.startswith("offset:")), None))
                lgkm[int(ops[0][1:])] = lds[:, j].copy()
            elif op in ("buffer_load_dword", "buffer_load_sshort", "buffer_load_sbyte"):
                size = {"buffer_load_dword": 4, "buffer_load_sshort": 2, "buffer_load_sbyte": 1}[op]
                arr, inr, idx = access(ops, size)
                assert arr.dtype.itemsize == (8 if size == 4 else size), "load width differs from the buffer's"
                d = int(ops[0][1:])
                assert d not in pending
                # narrow loads sign-extend (the buffers of int16 / int8 are kept in their own type)
                pending[d] = np.where(inr, arr[np.where(inr, idx, 0)].astype(np.int64), 0) & M32
            elif op in ("buffer_store_dword", "buffer_atomic_add"):
                assert not pending and not lgkm, "store with loads in flight"
                arr, inr, idx = access(ops)
                assert arr is y
                v = val(ops[0]).astype(np.int64)
                if op == "buffer_store_dword":
                    assert not atomic_ok
                    y[idx[inr]] = v[inr]
                else:
                    assert atomic_ok
                    np.add.at(y, idx[inr], v[inr])
                    y &= M32
                for t in idx[inr]:
                    stored[int(t)] += 1
            elif op == "v_mov_b32_e32":
                V[int(ops[0][1:])] = np.broadcast_to(val(ops[1]), V[4].shape).astype(np.int64)
            elif op in ("v_add_u32_e32", "v_sub_u32_e32"):
                a, b = np.int64(0) + val(ops[1]), np.int64(0) + val(ops[2])
                V[int(ops[0][1:])] = ((a + b) if op == "v_add_u32_e32" else (a - b)) & M32
            elif op == "v_ashrrev_i32_e32":
                x = val(ops[2]).astype(np.int64)
                x = np.where(x >= 2 ** 31, x - 2 ** 32, x)
                V[int(ops[0][1:])] = (x >> int(ops[1], 0)) & M32
            elif op == "v_max_i32_e32":
                a = val(ops[2]).astype(np.int64)
                sa = np.where(a >= 2 ** 31, a - 2 ** 32, a)
                V[int(ops[0][1:])] = np.maximum(sa, int(ops[1], 0)) & M32
            elif op in ("v_mul_lo_u32", "v_mul_hi_i32"):
                a = val(ops[1])
                sa = a - 2 ** 32 if a >= 2 ** 31 else a
                b = val(ops[2]).astype(np.int64)
                sb = np.where(b >= 2 ** 31, b - 2 ** 32, b).astype(object)
                p = sb * sa
                V[int(ops[0][1:])] = np.array(((p & M32) if op == "v_mul_lo_u32" else ((p >> 32) & M32)),
                                              dtype=np.int64)
            elif op == "v_mad_i32_i24":
                def s24(t):
                    t = np.asarray(t, dtype=np.int64) & 0xFFFFFF
                    return np.where(t >= 2 ** 23, t - 2 ** 24, t)
                p_ = s24(val(ops[1])) * s24(val(ops[2])) + val(ops[3])
                V[int(ops[0][1:])] = np.asarray(p_, dtype=np.int64) & M32
            elif op == "v_alignbit_b32":
                hi, lo = val(ops[1]).astype(object), val(ops[2]).astype(object)
                sh = int(ops[3], 0)
                V[int(ops[0][1:])] = np.array((((hi << 32) | lo) >> sh) & M32, dtype=np.int64)
            elif op == "s_endpgm":
                assert not lgkm
                return
            elif op == "s_nop":
                pass
            else:
                raise AssertionError(f"unexpected instruction {op} at {pc:#x}")
            pc = nxt


def to_i32(a):
    a = np.asarray(a, dtype=np.int64) & M32
    return np.where(a >= 2 ** 31, a - 2 ** 32, a).astype(np.int32)


CASES = [
    # n, c, h, w, k, r, s, stride, pad, splits, epilogue
    (2, 5, 9, 9, 70, 3, 3, 1, 1, 1, "full"),
    (2, 5, 9, 9, 70, 3, 3, 2, 1, 2, "none"),
    (3, 7, 12, 12, 64, 1, 1, 1, 0, 1, "relu"),
    (1, 6, 7, 8, 20, 2, 3, 1, 1, 3, "full"),
    (1, 3, 10, 10, 5, 3, 3, 2, 0, 1, "mul"),
    (33, 40, 1, 1, 17, 1, 1, 1, 0, 1, "full"),     # a LinearShift [33 x 40] -> 17 (on x^T)
    (1, 70, 1, 1, 20, 1, 1, 1, 0, 2, "full"),      # a LinearShift of one row (on x)
    (2, 64, 4, 4, 3, 3, 3, 1, 1, 4, "full"),
    (2, 3, 13, 11, 70, 7, 7, 2, 3, 1, "full"),     # a padded copy of x (windows over 3 x 3)
    (1, 4, 9, 10, 20, 5, 4, 1, 2, 2, "none"),
    (1, 2, 12, 12, 9, 4, 6, 3, 0, 1, "relu"),      # stride leaves the last rows unread
    # wave splits (forced): 2 or 4 waves share 64 pixels, each with a share of
    # the reduction, meeting in LDS
    (2, 40, 9, 9, 70, 3, 3, 1, 1, 1, "full", 2),
    (3, 37, 7, 6, 64, 3, 3, 2, 1, 1, "full", 4),
    (2, 5, 9, 9, 33, 3, 3, 1, 1, 2, "none", 4),     # with split-K: atomics of each share
    (1, 300, 3, 5, 130, 1, 1, 1, 0, 1, "mul", 4),
    (1, 3, 13, 11, 20, 7, 7, 2, 3, 1, "relu", 2),   # padded copy and wave split
    # splits of 8 and 16 waves (workgroups of 512 / 1024 threads), and segments
    # of 16 or 32 output channels
    (2, 40, 9, 9, 70, 3, 3, 1, 1, 1, "full", 8),
    (1, 300, 3, 5, 130, 1, 1, 1, 0, 1, "full", 16),
    (2, 37, 7, 6, 70, 3, 3, 2, 1, 2, "none", 16),   # with split-K
    (2, 40, 9, 9, 70, 3, 3, 1, 1, 1, "full", 1, 16),
    (2, 13, 9, 9, 50, 3, 3, 1, 1, 3, "none", 4, 32),
    (33, 90, 1, 1, 37, 1, 1, 1, 0, 1, "full", 16, 16),
    (1, 3, 13, 11, 40, 7, 7, 2, 3, 1, "relu", 8, 16),  # padded copy
    # several groups of 64 pixels per workgroup, each with a wave split
    (2, 40, 9, 9, 70, 3, 3, 1, 1, 1, "full", 4, 64, 4),   # 16 waves: 4 groups x 4 shares
    (33, 300, 1, 1, 130, 1, 1, 1, 0, 2, "none", 4, 64, 4),
    (2, 37, 7, 6, 70, 3, 3, 2, 1, 1, "full", 8, 32, 2),
    (3, 13, 9, 9, 50, 3, 3, 1, 1, 1, "relu", 1, 64, 1),   # one wave per workgroup
    (1, 3, 13, 11, 40, 7, 7, 2, 3, 1, "mul", 2, 16, 4),   # padded copy
]


LINEAR_CASES = [
    # n, c, h, w, k, r, s, stride, pad, splits, epilogue, wave split, channels, pixel groups
    (33, 40, 1, 1, 17, 1, 1, 1, 0, 1, "full", 1, 64, None),
    (70, 300, 1, 1, 130, 1, 1, 1, 0, 2, "full", 4, 64, None),
    (130, 90, 1, 1, 70, 1, 1, 1, 0, 1, "relu", 16, 16, 1),
    (65, 200, 1, 1, 33, 1, 1, 1, 0, 3, "none", 2, 32, 4),
]


@pytest.mark.parametrize("transpose", [0, 1])
@pytest.mark.parametrize("case", LINEAR_CASES, ids=[str(i) for i in range(len(LINEAR_CASES))])
def test_linear_plans_on_x_and_on_x_transposed(case, transpose, tmp_path, knob):
    knob("DS_JIT_TRANSPOSE", transpose)
    run_generated(case, zlib.crc32(str((case, transpose)).encode()), 0.1, tmp_path, knob)


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_generated_code_matches_oracle(case, tmp_path, knob):
    wsplit = case[11] if len(case) > 11 else 1
    tn = case[12] if len(case) > 12 else 64
    pgroups = case[13] if len(case) > 13 else None
    run_generated(case[:11] + (wsplit, tn, pgroups), zlib.crc32(str(case).encode()), 0.1, tmp_path, knob)


def random_cases(count, seed=1905):
    """Seeded random shapes: windows 1-5 (over 3 x 3: padded copies), strides 1-3,
    padding 0-2, ragged channel counts, forced splits and wave splits, every
    epilogue, weight sparsity from none to 95 % (whole elements without a
    non-zero weight, which are skipped)."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        n, c, k = int(rng.integers(1, 4)), int(rng.integers(1, 80)), int(rng.integers(1, 150))
        r, s = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        st, pd = int(rng.integers(1, 4)), int(rng.integers(0, 3))
        h, w = int(rng.integers(max(1, r - 2 * pd), 12)), int(rng.integers(max(1, s - 2 * pd), 12))
        if h + 2 * pd < r or w + 2 * pd < s:
            continue
        splits = int(rng.choice([1, 2, 3]))
        wsplit = int(rng.choice([1, 2, 4, 8, 16]))
        tn = int(rng.choice([16, 32, 64, 64]))
        epi = str(rng.choice(["none", "relu", "mul", "full"]))
        zero = float(rng.choice([0.0, 0.1, 0.5, 0.95]))
        pg = int(rng.choice([p for p in (1, 2, 4) if p * wsplit <= 16]))
        out.append(((n, c, h, w, k, r, s, st, pd, splits, epi, wsplit, tn, pg), zero))
    return out


RANDOM = random_cases(20)


@pytest.mark.parametrize("case,zero", RANDOM, ids=[str(i) for i in range(len(RANDOM))])
def test_generated_code_matches_oracle_random_shapes(case, zero, tmp_path, knob):
    run_generated(case, zlib.crc32(repr((case, zero)).encode()), zero, tmp_path, knob)


def run_generated(case, seed, zero_frac, tmp_path, knob):
    """Generate a plan's code object for `case` (n, c, h, w, k, r, s, stride, pad,
    splits, epilogue, wave split, channels per segment), run it in the
    interpreter over every lane, and compare with the oracle."""
    n, c, h, w, k, r, s, st, pd, splits, epi, wsplit, tn, pgroups = case
    knob("DS_JIT_WSPLIT", wsplit)
    knob("DS_JIT_TN", tn)
    knob("DS_JIT_PGROUPS", pgroups or -1)
    codes, x, rng = gen_layer(seed, n, c, h, w, k, r, s, zero_frac)
    bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
    mul = add = res = None
    relu = epi in ("full", "relu")
    if epi in ("full", "mul"):
        mul = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
        add = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
        add[0] = 0
    wp = ops.pack_shift_weights(codes)
    lanes, (oh, ow) = plan_lanes(n, c, h, w, k, r, s, st, pd, wsplit, pgroups)
    if epi == "full":
        res = rng.integers(-(2 ** 31), 2 ** 31, (n, k, oh, ow), dtype=np.int64).astype(np.int32)
    img = ops.jit_conv_image(wp, (n, c, h, w), (r, s), st, pd, bias=bias, mul=mul, add=add,
                             mul_shift=13, residual=res is not None, relu=relu, splits=splits)

    loads, addr, off, size = elf_layout(img)
    assert max(int(ld[2], 16) for ld in loads) == addr          # highest loadable segment
    assert [ld for ld in loads if int(ld[2], 16) == addr][0][1] == f"0x{off:06x}"
    assert off + size == len(img)

    insts = disassemble(img, str(tmp_path))
    body = min(insts)
    # Layers with one tap per element run the 80-VGPR entry point, which hands
    # over v3, v4 and v13 only: v5..v12 must be written before they are read.
    one_tap = r * s == 1 or r > 3 or s > 3
    if one_tap:
        for i in range(5, 13):
            del lanes[i]
    top = max(int(t[1:]) for _, ops_, _ in insts.values() for t in ops_ if re.fullmatch(r"v\d+", t))
    assert top < (80 if one_tap else 96), f"v{top} is outside the entry point's registers"
    conv = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    xb, xbytes = x_buffer(x, r, s, st, pd)
    y = np.full(n * k * oh * ow, 0xDEADBEEF, dtype=np.int64)
    bufs = {20: (xb, xbytes), 24: (y, y.size * 4)}
    bufs[36] = (res.reshape(-1).view(np.uint32).astype(np.int64), y.size * 4) if res is not None else (y, 0)
    nsplit = min(splits, c)
    kgroups = -(-k // tn)
    split = nsplit > 1
    tr = transposed_linear(n, h, w, r, s)
    if tr:      # the kernel reads no residual (the last pass adds it)
        bufs[36] = (y, 0)
    if split:
        y[:] = y_start(bias, n, k, oh, ow, tr)
    stubs = sum(1 for op, _, _ in insts.values() if op == "s_getpc_b64")
    assert stubs == kgroups * nsplit * wsplit
    interp = Interp(insts, bufs, wsplit, pgroups)
    total = collections.Counter()
    for seg in range(kgroups * nsplit):
        # the waves of one pixel group: each share up to the barrier, then each to the end
        lds = np.zeros((lanes[4].size, 64), np.int64)
        runs = [interp.run(body + 20 * (seg * wsplit + sh), seg * wsplit + sh, lanes, y, split, lds, total)
                for sh in range(wsplit)]
        for _ in range(2 if wsplit > 1 else 1):
            for r_ in runs:
                next(r_, None)
        for r_ in runs:
            assert next(r_, "done") == "done", "a second barrier"
    assert len(total) == y.size and set(total.values()) == {nsplit}
    if tr:
        y = transpose_back(y, n, k, None if split else res, relu and not split)
    got = to_i32(y).reshape(n, k, oh, ow)
    if split:
        np.testing.assert_array_equal(got, conv)
    else:
        want = oracle.epilogue(conv, mul, add, 13, residual=res, relu=relu)
        np.testing.assert_array_equal(got, want)


def test_image_rejects_bad_arguments():
    codes = np.full((4, 9), 15, np.uint8)
    wp = ops.pack_shift_weights(codes)
    with pytest.raises(ops.DeepShiftError, match="UNSUPPORTED"):
        ops.jit_conv_image(ops.pack_shift_weights(np.full((4, 1024), 15, np.uint8)), (1, 1, 1, 1100),
                           (1, 1024))
    with pytest.raises(ops.DeepShiftError, match="INVALID_SHAPE"):
        ops.jit_conv_image(wp, (1, 1, 2, 2), 3)
    with pytest.raises(ops.DeepShiftError, match="INVALID_ARG"):
        ops.jit_conv_image(wp, (1, 1, 8, 8), 3, add=np.zeros(4, np.int32))
    with pytest.raises(ops.DeepShiftError, match="INVALID_ARG"):
        ops.jit_conv_image(wp, (1, 1, 8, 8), 3, mul=np.ones(4, np.int32), mul_shift=32)
    bad = wp.copy()
    bad[0, 0] |= 1 << 30
    with pytest.raises(ops.DeepShiftError, match="INVALID_CODE"):
        ops.jit_conv_image(bad, (1, 1, 8, 8), 3)


def test_zero_weights_emit_no_arithmetic(tmp_path):
    """A segment whose weights are all zero is bias and stores only: elements with
    no non-zero weight in a segment are not even loaded."""
    codes = np.full((8, 4), 15 | 16, np.uint8)
    img = ops.jit_conv_image(ops.pack_shift_weights(codes), (1, 4, 3, 3), 1, splits=1)
    names = collections.Counter(op for op, _, _ in disassemble(img, str(tmp_path)).values())
    assert names["v_add_u32_e32"] == names["v_sub_u32_e32"] == names["v_ashrrev_i32_e32"] == 0
    assert names["buffer_load_dword"] == 0 and names["buffer_store_dword"] == 8
    codes[3, 2] = 16 | 4      # one non-zero weight: one load, one shift, one subtract
    img = ops.jit_conv_image(ops.pack_shift_weights(codes), (1, 4, 3, 3), 1, splits=1)
    names = collections.Counter(op for op, _, _ in disassemble(img, str(tmp_path)).values())
    assert names["buffer_load_dword"] == 1 and names["v_ashrrev_i32_e32"] == 1
    assert names["v_sub_u32_e32"] == 1 and names["v_add_u32_e32"] == 0


def test_small_grids_run_unsplit_in_16_channel_segments(tmp_path, knob):
    """A grid of a few waves whose default plan would split the reduction runs
    unsplit in segments of 16 channels with a wave split of 8 (24 waves at a split
    of 4 double to 48; no fill pass, no atomics): the same code as that
    configuration forced, and correct."""
    codes, _, _ = gen_layer(7, 1, 32, 10, 10, 40, 3, 3)
    wp = ops.pack_shift_weights(codes)
    auto = ops.jit_conv_image(wp, (1, 32, 10, 10), 3, 1, 1)
    names = collections.Counter(op for op, _, _ in disassemble(auto, str(tmp_path)).values())
    assert names["s_getpc_b64"] == 3 * 8 and names["buffer_atomic_add"] == 0
    knob("DS_JIT_TN", 16)
    knob("DS_JIT_WSPLIT", 8)
    assert ops.jit_conv_image(wp, (1, 32, 10, 10), 3, 1, 1, splits=1) == auto
    knob("DS_JIT_TN", 64)     # segments of 64 forced: the split plan of the older rule
    knob("DS_JIT_WSPLIT", -1)
    old = ops.jit_conv_image(wp, (1, 32, 10, 10), 3, 1, 1)
    names = collections.Counter(op for op, _, _ in disassemble(old, str(tmp_path)).values())
    assert names["buffer_atomic_add"] > 0
    run_generated((1, 32, 10, 10, 40, 3, 3, 1, 1, 1, "full", 8, 16, 1), 7, 0.1, tmp_path, knob)


def test_small_grids_of_several_tiles_split_in_two(tmp_path, knob):
    """Four or more pixel tiles sharing each code stream, one workgroup per CU
    twice over: 16-channel segments in 2 parts (fill pass and atomics), the code
    of that configuration forced."""
    codes, _, _ = gen_layer(8, 1, 64, 20, 20, 64, 3, 3)
    wp = ops.pack_shift_weights(codes)
    auto = ops.jit_conv_image(wp, (1, 64, 20, 20), 3, 1, 1)
    names = collections.Counter(op for op, _, _ in disassemble(auto, str(tmp_path)).values())
    # 7 tiles of 64 pixels x 4 groups of 16 channels; about 60 KiB of code per
    # group, so a wave split of 8 (7.5 KiB per wave)
    knob("DS_JIT_TN", 16)
    knob("DS_JIT_WSPLIT", 8)
    assert ops.jit_conv_image(wp, (1, 64, 20, 20), 3, 1, 1, splits=2) == auto
    assert names["s_getpc_b64"] == 4 * 2 * 8 and names["buffer_atomic_add"] > 0


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_code_width_does_not_change_the_generated_code(bits):
    """The generated code depends on the weights only: b-bit packed codes give the
    same code object as the same weights in the 5-bit format."""
    rng = np.random.default_rng(bits)
    ones = (1 << (bits - 1)) - 1
    shift = rng.integers(0, ones, (70, 5 * 9))
    shift[rng.random(shift.shape) < 0.2] = 15
    codes = (rng.integers(0, 2, shift.shape) << 4 | shift).astype(np.uint8)
    bias = rng.integers(-1000, 1000, 70).astype(np.int32)
    a = ops.jit_conv_image(ops.pack_shift_weights(codes), (2, 5, 9, 9), 3, 1, 1, bias=bias)
    b = ops.jit_conv_image(ops.pack_shift_weights(codes, bits=bits), (2, 5, 9, 9), 3, 1, 1, bias=bias,
                           code_bits=bits)
    assert a == b



MUL_CASES = [
    # n, c, h, w, k, r, s, stride, pad, splits, wave split, zero fraction
    (2, 5, 9, 9, 70, 3, 3, 1, 1, 1, 1, 0.1),
    (2, 5, 9, 9, 70, 3, 3, 2, 1, 2, 1, 0.3),
    (3, 7, 12, 12, 64, 1, 1, 1, 0, 1, 4, 0.0),
    (33, 40, 1, 1, 17, 1, 1, 1, 0, 2, 2, 0.5),
    (1, 3, 13, 11, 20, 7, 7, 2, 3, 1, 1, 0.1),
]


@pytest.mark.parametrize("case", MUL_CASES, ids=[str(i) for i in range(len(MUL_CASES))])
def test_multiplication_plan_matches_oracle(case, tmp_path, knob):
    """Multiplication plans (the comparison operator in the plans' tiling): one
    v_mad_i32_i24 per non-zero weight, weights as inline constants or s_mov_b32
    literals; run in the interpreter against the oracle's 24-bit product."""
    n, c, h, w, k, r, s, st, pd, splits, wsplit, zero = case
    knob("DS_JIT_WSPLIT", wsplit)
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    wt = rng.integers(-(2 ** 23), 2 ** 23, (k, c * r * s)).astype(np.int32)
    small = rng.random(wt.shape) < 0.3
    wt[small] = rng.integers(-16, 65, int(small.sum()))        # inline-constant weights
    wt[rng.random(wt.shape) < zero] = 0
    x = rng.integers(-(2 ** 31), 2 ** 31, (n, c, h, w), dtype=np.int64).astype(np.int32)
    bias = rng.integers(-(2 ** 31), 2 ** 31, k, dtype=np.int64).astype(np.int32)
    img = ops.jit_conv_mul_image(wt, (n, c, h, w), (r, s), st, pd, bias=bias, splits=splits)
    insts = disassemble(img, str(tmp_path))
    names = collections.Counter(op for op, _, _ in insts.values())
    body = min(insts)
    lanes, (oh, ow) = plan_lanes(n, c, h, w, k, r, s, st, pd, wsplit)
    one_tap = r * s == 1 or r > 3 or s > 3
    if one_tap:
        for i in range(5, 13):
            del lanes[i]
    xb, xbytes = x_buffer(x, r, s, st, pd)
    y = np.full(n * k * oh * ow, 0xDEADBEEF, dtype=np.int64)
    bufs = {20: (xb, xbytes), 24: (y, y.size * 4), 36: (y, 0)}
    nsplit = min(splits, c)
    tr = transposed_linear(n, h, w, r, s)
    if nsplit > 1:
        y[:] = y_start(bias, n, k, oh, ow, tr)
    interp = Interp(insts, bufs, wsplit)
    total = collections.Counter()
    for seg in range(-(-k // 64) * nsplit):
        lds = np.zeros((lanes[4].size, 64), np.int64)
        runs = [interp.run(body + 20 * (seg * wsplit + sh), seg * wsplit + sh, lanes, y, nsplit > 1, lds, total)
                for sh in range(wsplit)]
        for _ in range(2 if wsplit > 1 else 1):
            for r_ in runs:
                next(r_, None)
        for r_ in runs:
            assert next(r_, "done") == "done"
    if tr:
        y = transpose_back(y, n, k)
    want = oracle.conv2d_mul24(x, wt, bias, r=r, s=s, stride=st, pad=pd)
    np.testing.assert_array_equal(to_i32(y).reshape(want.shape), want)
    # exactly one v_mad_i32_i24 per non-zero weight, no shift-plan arithmetic
    assert names["v_mad_i32_i24"] == int(np.sum(wt != 0))
    assert names["v_add_u32_e32"] == names["v_sub_u32_e32"] == names["v_ashrrev_i32_e32"] == 0



@pytest.mark.parametrize("act_bits", [16, 8])
@pytest.mark.parametrize("case", [(2, 5, 9, 9, 70, 3, 3, 1, 1, 1, 1), (3, 7, 12, 12, 64, 1, 1, 2, 0, 2, 2),
                                  (1, 3, 13, 11, 20, 7, 7, 2, 3, 1, 1), (9, 40, 1, 1, 17, 1, 1, 1, 0, 1, 4)],
                         ids=["3x3", "1x1s2_split", "stem_padded", "linear"])
def test_narrow_activation_plans_match_oracle(case, act_bits, tmp_path, knob):
    """Plans with int16 / int8 activations: sign-extending narrow loads of x (the
    padded copy of wide windows is int32), the same arithmetic as int32 plans;
    against the oracle on the sign-extended inputs."""
    n, c, h, w, k, r, s, st, pd, splits, wsplit = case
    knob("DS_JIT_WSPLIT", wsplit)
    codes, _, rng = gen_layer(zlib.crc32(repr((case, act_bits)).encode()), n, c, h, w, k, r, s, 0.1)
    dt = {16: np.int16, 8: np.int8}[act_bits]
    info = np.iinfo(dt)
    x = rng.integers(info.min, info.max, (n, c, h, w), endpoint=True).astype(dt)
    bias = rng.integers(-(2 ** 20), 2 ** 20, k).astype(np.int32)
    img = ops.jit_conv_image(ops.pack_shift_weights(codes), (n, c, h, w), (r, s), st, pd, bias=bias,
                             splits=splits, act_bits=act_bits)
    insts = disassemble(img, str(tmp_path))
    names = collections.Counter(op for op, _, _ in insts.values())
    ext = padded_extents(h, w, r, s, st, pd)
    # x itself is read narrow; the padded and transposed copies are int32
    narrow = ext is None and not transposed_linear(n, h, w, r, s)
    narrow_op = {16: "buffer_load_sshort", 8: "buffer_load_sbyte"}[act_bits]
    if narrow:
        assert names[narrow_op] > 0 and names["buffer_load_dword"] == 0
    else:
        assert names[narrow_op] == 0 and names["buffer_load_dword"] > 0
    body = min(insts)
    lanes, (oh, ow) = plan_lanes(n, c, h, w, k, r, s, st, pd, wsplit)
    if narrow:            # the template scales tap offsets by the element size
        for i in range(4, 13):
            lanes[i] = np.where(lanes[i] == OOB, OOB, lanes[i] // 4 * x.itemsize)
    if r * s == 1 or r > 3 or s > 3:
        for i in range(5, 13):
            del lanes[i]
    if narrow:
        xb = np.ascontiguousarray(x).reshape(-1)
        bufs = {20: (xb, xb.size * x.itemsize)}
    else:
        xb, xbytes = x_buffer(x.astype(np.int32), r, s, st, pd)
        bufs = {20: (xb, xbytes)}
    y = np.full(n * k * oh * ow, 0xDEADBEEF, dtype=np.int64)
    bufs[24] = (y, y.size * 4)
    bufs[36] = (y, 0)
    nsplit = min(splits, c)
    tr = transposed_linear(n, h, w, r, s)
    if nsplit > 1:
        y[:] = y_start(bias, n, k, oh, ow, tr)
    interp = Interp(insts, bufs, wsplit)
    total = collections.Counter()
    for seg in range(-(-k // 64) * nsplit):
        lds = np.zeros((lanes[4].size, 64), np.int64)
        runs = [interp.run(body + 20 * (seg * wsplit + sh), seg * wsplit + sh, lanes, y, nsplit > 1, lds, total)
                for sh in range(wsplit)]
        for _ in range(2 if wsplit > 1 else 1):
            for r_ in runs:
                next(r_, None)
        for r_ in runs:
            assert next(r_, "done") == "done"
    if tr:
        y = transpose_back(y, n, k)
    want = oracle.conv2d_shift(x, codes, bias, r=r, s=s, stride=st, pad=pd)
    np.testing.assert_array_equal(to_i32(y).reshape(want.shape), want)
