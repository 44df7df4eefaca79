"""Sanitizer tier (CPU only): the oracle and the ABI's host-side code built
with AddressSanitizer and UndefinedBehaviorSanitizer.

* The oracle (oracle/mhlmoe_oracle.c) is compiled with
  -fsanitize=address,undefined and every pin of tests/oracle_pins.py runs
  against it in a child process (the ASan runtime preloaded, since the
  Python interpreter itself is not instrumented).  Any out-of-bounds access,
  use after free, signed overflow or misaligned load aborts the child.
* The ABI's own source (csrc/api.cpp: argument validation, workspace layout,
  the entry points' early returns) is compiled with the same sanitizers into
  tests/host_abi_check.cpp's driver, with the kernel launchers replaced by
  stubs that abort; the driver sizes the workspace of every entry point over
  a table of valid, boundary and invalid shapes, and the sizes must equal
  those of the production library.  Nothing here touches a GPU.
"""
import os
import re
import shutil
import subprocess
import sys

import pytest

import oracle
import paper_2602_04870_amd as mh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_04870_amd", "csrc")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _gcc_runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip(f"gcc has no {name}")
    return path


PINS_CHILD = r"""
import sys
sys.path.insert(0, {root!r})
import oracle
from tests import oracle_pins
o = oracle.Oracle(oracle.load({lib!r}))
for pin in oracle_pins.ALL_PINS:
    pin(o)
    print("pin ok", pin.__name__, flush=True)
print("ALL PINS PASSED", flush=True)
"""


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    oracle.compile_library(oracle.SOURCE, lib, flags=SAN)
    env = dict(os.environ, OMP_NUM_THREADS="4", LD_PRELOAD=_gcc_runtime("libasan.so"),
               **SAN_ENV)
    res = subprocess.run([sys.executable, "-c", PINS_CHILD.format(root=ROOT, lib=lib)],
                         capture_output=True, text=True, timeout=900, env=env)
    out = res.stdout + res.stderr
    assert res.returncode == 0 and "ALL PINS PASSED" in res.stdout, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]


def _stubs(path):
    """Definitions of every kernel launcher declared in launch.hpp that abort
    when called (the driver must never get as far as a launch)."""
    text = open(os.path.join(CSRC, "launch.hpp")).read()
    decls = re.findall(r"^hipError_t\s+(\w+)\(([^;{]*)\);", text, flags=re.M)
    assert len(decls) >= 14, decls
    body = ['#include <cstdio>', '#include <cstdlib>', '#include "launch.hpp"', "namespace mhl {"]
    for name, params in decls:
        body.append(f"hipError_t {name}({params}) {{ std::fprintf(stderr, \"launch {name}\\n\"); "
                    "std::abort(); }")
    body.append("}  // namespace mhl")
    open(path, "w").write("\n".join(body) + "\n")


def test_abi_host_code_under_asan_ubsan(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no g++")
    stubs = str(tmp_path / "stubs.cpp")
    _stubs(stubs)
    exe = str(tmp_path / "host_abi_check")
    inc = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT}/include", f"-I{CSRC}",
           "-Wno-unused-result", "-Wno-unused-value", "-Wno-attributes"]
    cmd = [gxx, "-std=c++17", *SAN, *inc, os.path.join(CSRC, "api.cpp"), stubs,
           os.path.join(ROOT, "tests", "host_abi_check.cpp"), "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, **SAN_ENV))
    out = res.stdout + res.stderr
    assert res.returncode == 0 and "done 0 failures" in res.stdout, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    # the sanitized host code sizes workspaces exactly as the production library
    lib = mh.load_library()
    import ctypes
    n = 0
    for line in res.stdout.splitlines():
        if not line.startswith("ws "):
            continue
        op, T, Nh, dh, Ne, k, dff, dt, st, nbytes = (int(v) for v in line.split()[1:])
        b = ctypes.c_size_t(0)
        st2 = lib.mhlmoe_workspace_size(op, T, Nh, dh, Ne, k, dff, dt, ctypes.byref(b))
        assert st2 == st, line
        if st == 0:
            assert b.value == nbytes, line
        n += 1
    assert n > 500
