"""CPU sanitizer pass: the oracle and the library's host code under
AddressSanitizer and UndefinedBehaviorSanitizer.

* The oracle (oracle.c) is built with gcc -fsanitize=address,undefined and its
  pins run against that build.
* The library is built with the host compilation of every source sanitized
  (hipcc -Xarch_host -fsanitize=...; device code as usual) and the CPU tests of
  its host code run against it: argument validation of every entry point, the
  packers, and the plan code generator (ds_jit_conv_image, through the
  interpreter of test_jit_codegen).

Each run is a subprocess with the sanitizer runtime preloaded (the Python
interpreter itself is not instrumented) and stops at the first report.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1",
       "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}

pytestmark = pytest.mark.slow


def run(preload, bootstrap, tests):
    code = ("import sys; sys.path.insert(0, %r)\n%s\nimport pytest\n"
            "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider'] + %r))" % (ROOT, bootstrap, tests))
    env = dict(os.environ, **ENV, LD_PRELOAD=preload)
    res = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=900)
    assert res.returncode == 0, (res.stdout[-3000:] + res.stderr[-6000:])
    return res.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fno-omit-frame-pointer", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-o", lib,
                    os.path.join(ROOT, "oracle", "oracle.c")], check=True)
    rt = ":".join(subprocess.run(["gcc", f"-print-file-name={n}"], capture_output=True, text=True,
                                 check=True).stdout.strip() for n in ("libasan.so", "libubsan.so"))
    boot = ("import oracle\noracle._LIB = %r\nassert oracle._load()._name == %r" % (lib, lib))
    out = run(rt, boot, ["tests/test_oracle_pins.py", "tests/test_oracle_layer_pins.py",
                         "tests/test_oracle_convert_pins.py", "tests/test_oracle_backward_pins.py",
                         "tests/test_oracle_bits_pins.py", "tests/test_oracle_narrow_pins.py",
                         "tests/test_oracle_network_pins.py"])
    assert "passed" in out


def test_library_host_code_under_asan_ubsan():
    from paper_1905_13298_amd import build
    lib = build.build(sanitize=True)
    (rt,) = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    boot = ("from paper_1905_13298_amd import build, _native\nbuild.LIB = %r\n"
            "assert _native.lib()._name == %r" % (lib, lib))
    out = run(rt, boot, ["tests/test_abi_cpu.py", "tests/test_jit_codegen.py", "tests/test_oracle_bits_pins.py"])
    assert "passed" in out
