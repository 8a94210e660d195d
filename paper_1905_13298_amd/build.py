"""Build ``libdeepshift.so`` (the C-ABI library) in-tree for gfx950.

HIP sources go through hipcc for gfx950 with packed-FP32 instructions
disabled; host-only sources go through g++. Objects are written to
``_build/`` next to this file and linked into ``libdeepshift.so``.
"""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
INCLUDE = os.path.join(ROOT, "include")
CSRC = os.path.join(PKG, "csrc")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdeepshift.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-Wall",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", INCLUDE, "-I", CSRC]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-I", INCLUDE, "-I", CSRC]

HIP_SOURCES = ["shift_ops.hip", "conv_kernels.hip", "convert.hip", "pool.hip", "jit.hip", "backward.hip"]
CXX_SOURCES = ["pack.cpp", "tuning.cpp"]
LLVM = "/opt/rocm/llvm/bin"

# The weight-specialised kernel template (jit_template.hip) is compiled to
# gfx950 assembly; the JITBODY marker of each of its two kernels becomes a jump
# through a table at the start of section .jitbody, indexed by the segment
# number in s19 (stubs of 20 bytes each). The table and the segments' code are
# generated at run time.
JIT_JUMP = """s_getpc_b64 s[28:29]
	s_add_u32 s28, s28, ds_jit_body@rel32@lo+4
	s_addc_u32 s29, s29, ds_jit_body@rel32@hi+12
	s_mul_i32 s30, s19, 20
	s_add_u32 s28, s28, s30
	s_addc_u32 s29, s29, 0
	s_setpc_b64 s[28:29]"""
JIT_BODY_SECTION = """
	.section .jitbody,"ax",@progbits
	.p2align 8
	.hidden ds_jit_body
	.globl ds_jit_body
ds_jit_body:
	.fill 64, 4, 0xbf810000
"""


# Host-code sanitizers (AddressSanitizer, UndefinedBehaviorSanitizer) for a CPU
# check of the library's host code -- the code generator, packer and argument
# checks. Each -fsanitize= applies to the host compilation only (-Xarch_host);
# device code is built as usual. The result is a separate library that only the
# CPU tests load, with the clang ASan runtime preloaded.
SAN_HOST = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
            "-fno-omit-frame-pointer"]
CLANGXX = os.path.join(os.path.dirname(HIPCC), "..", "llvm", "bin", "clang++")


def _compile(src: str, objdir: str = OBJDIR, sanitize: bool = False) -> str:
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    path = os.path.join(CSRC, src)
    if src.endswith(".hip"):
        san = [t for f in SAN_HOST for t in ("-Xarch_host", f)] if sanitize else []
        cmd = [HIPCC, *HIP_FLAGS, *san, "-c", path, "-o", obj]
    elif sanitize:
        cmd = [CLANGXX, *CXX_FLAGS, *SAN_HOST, "-c", path, "-o", obj]
    else:
        cmd = ["g++", *CXX_FLAGS, "-c", path, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")


def _jit_template() -> str:
    """Build the template code object and an x86 object that embeds it
    (symbols ds_jit_template_image / ds_jit_template_image_end)."""
    src = os.path.join(CSRC, "jit_template.hip")
    asm = os.path.join(OBJDIR, "jit_template.s")
    _run([HIPCC, *HIP_FLAGS, "--cuda-device-only", "-S", src, "-o", asm])
    text = open(asm).read()
    marker = "; JITBODY"
    if text.count(marker) != 2:
        raise RuntimeError("jit_template.s: expected a JITBODY marker in each of its two kernels")
    text = text.replace(marker, JIT_JUMP) + JIT_BODY_SECTION
    spliced = os.path.join(OBJDIR, "jit_template_spliced.s")
    with open(spliced, "w") as f:
        f.write(text)
    obj = os.path.join(OBJDIR, "jit_template_dev.o")
    hsaco = os.path.join(OBJDIR, "jit_template.hsaco")
    _run([os.path.join(LLVM, "clang"), "-target", "amdgcn-amd-amdhsa", f"-mcpu={ARCH}",
          "-c", spliced, "-o", obj])
    _run([os.path.join(LLVM, "ld.lld"), "-shared", obj, "-T",
          os.path.join(CSRC, "jit_template.ld"), "-o", hsaco])
    embed = os.path.join(OBJDIR, "jit_image.S")
    with open(embed, "w") as f:
        f.write(f"""\t.section .rodata
\t.balign 64
\t.globl ds_jit_template_image
\t.hidden ds_jit_template_image
ds_jit_template_image:
\t.incbin "{hsaco}"
\t.globl ds_jit_template_image_end
\t.hidden ds_jit_template_image_end
ds_jit_template_image_end:
\t.section .note.GNU-stack,"",@progbits
""")
    out = os.path.join(OBJDIR, "jit_image.o")
    _run(["gcc", "-c", embed, "-o", out])
    return out


def build(verbose: bool = False, sanitize: bool = False, out: str | None = None) -> str:
    """Compile every source and link the library; returns its path. sanitize: the
    host-sanitizer build (SAN_HOST) into `out` (objects in a directory of its own)."""
    objdir = OBJDIR if not sanitize else os.path.join(OBJDIR, "san")
    target = out or (LIB if not sanitize else os.path.join(objdir, "libdeepshift_san.so"))
    os.makedirs(objdir, exist_ok=True)
    srcs = HIP_SOURCES + CXX_SOURCES
    with ThreadPoolExecutor(len(srcs) + 1) as ex:
        jit = ex.submit(_jit_template)
        objs = list(ex.map(lambda f: _compile(f, objdir, sanitize), srcs)) + [jit.result()]
    tmp = target + f".tmp{os.getpid()}"
    san = [t for f in SAN_HOST[:2] for t in ("-Xarch_host", f)] + ["-shared-libsan"] if sanitize else []
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *san, "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, target)
    if verbose:
        print(f"built {target}")
    return target


def sources() -> list:
    return [os.path.join(CSRC, s) for s in HIP_SOURCES + CXX_SOURCES + ["jit_template.hip", "jit_template.ld"]] + \
        [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hpp", ".h"))] + \
        [os.path.join(INCLUDE, "deepshift.h")]


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(s) > t for s in sources())


if __name__ == "__main__":
    build(verbose=True)
