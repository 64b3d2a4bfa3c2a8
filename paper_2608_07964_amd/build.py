"""Build libeasybalance.so (and the input generator's libebsynth.so) for gfx950.

    python -m paper_2608_07964_amd.build        # or __graft_entry__.build()

Each translation unit is compiled by hipcc in parallel, then linked into a
shared library next to the Python binding.  No JIT, no torch extension: the
library exports a plain C ABI (include/easybalance.h).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libeasybalance.so")
SYNTH_SRC = os.path.join(ROOT, "synth", "fill.hip")
SYNTH_LIB = os.path.join(ROOT, "synth", "libebsynth.so")
SYNTH_HOST_SRC = os.path.join(ROOT, "synth", "gen_host.c")
SYNTH_HOST_LIB = os.path.join(ROOT, "synth", "libsynthhost.so")

SOURCES = ["api.cpp", "schedule.cpp", "pass.cpp", "route.hip", "permute.hip", "gemm.hip", "combine.hip",
           "sched_dev.hip", "noalloc.hip"]

ARCH = os.environ.get("EB_OFFLOAD_ARCH", "gfx950")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
COMMON = ["-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}",
          # packed fp32 VALU ops stay off (hipcc's host pass warns it does not
          # know the feature; that is harmless)
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function", "-Wno-unused-result"]


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{out}")
    if out.strip():
        print(out, file=sys.stderr)


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    _run([HIPCC, *COMMON, *lang, "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj])
    return obj


def build(verbose: bool = True) -> list[str]:
    os.makedirs(BUILD, exist_ok=True)
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs) + 1)) as ex:
        futs = [ex.submit(_compile, s) for s in srcs]
        fut_synth = ex.submit(_compile, SYNTH_SRC)
        objs = [f.result() for f in futs]
        synth_obj = fut_synth.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    tmp = SYNTH_LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", synth_obj, "-o", tmp])
    os.replace(tmp, SYNTH_LIB)
    # host generator: plain C, IEEE fp32 (no contraction, no fast-math)
    tmp = SYNTH_HOST_LIB + ".tmp"
    _run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off", SYNTH_HOST_SRC,
          "-o", tmp])
    os.replace(tmp, SYNTH_HOST_LIB)
    if verbose:
        print(f"built {LIB}, {SYNTH_LIB} ({ARCH}) and {SYNTH_HOST_LIB}")
    return [LIB, SYNTH_LIB, SYNTH_HOST_LIB]


if __name__ == "__main__":
    build()
