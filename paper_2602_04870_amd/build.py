"""Build libmhlmoe.so in-tree with hipcc for gfx950.

    python -m paper_2602_04870_amd.build          # build (parallel)
    python -m paper_2602_04870_amd.build --clean  # remove objects first

Objects go to ``_build/`` at the repository root; the shared library is
written next to this file, where the binding loads it from.
"""
from __future__ import annotations

import argparse
import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "mhlmoe")
LIBRARY = os.path.join(PKG, "libmhlmoe.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed fp32 instructions are disabled for every HIP translation unit.  MFMA
# accumulators are kept in ordinary VGPRs (the unified register file of
# gfx950), which avoids AGPR<->VGPR copies around the SwiGLU epilogue.
COMMON_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    f"-I{INCLUDE}", f"-I{CSRC}",
]

SOURCES = ["api.cpp", "route.hip", "route_64_bf16.hip", "route_64_f32.hip",
           "route_128_bf16.hip", "route_128_f32.hip", "bucket.hip", "experts.hip",
           "backward.hip", "projection.cpp", "static_scratch.hip"]
HEADERS = ["device_common.hpp", "ffn_common.hpp", "launch.hpp", "route_kernel.hpp", "sort_networks.hpp"]


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd.insert(1, "-xhip")
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    return obj


def build(clean: bool = False, jobs: int | None = None, verbose: bool = False) -> str:
    if clean and os.path.isdir(OBJDIR):
        shutil.rmtree(OBJDIR)
    os.makedirs(OBJDIR, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 1, 16)
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIBRARY + ".tmp%d" % os.getpid()
    rocm_lib = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(HIPCC))), "lib")
    # hipBLASLt for the dense projections of the latent layer.
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, f"-L{rocm_lib}",
           "-lhipblaslt", f"-Wl,-rpath,{rocm_lib}", "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIBRARY)
    if verbose:
        print(f"built {LIBRARY}")
    return LIBRARY


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--clean", action="store_true")
    ap.add_argument("-j", "--jobs", type=int, default=None)
    args = ap.parse_args(argv)
    build(clean=args.clean, jobs=args.jobs, verbose=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
