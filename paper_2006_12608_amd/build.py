"""Build libsj.so for gfx950 with hipcc (in-tree, next to this file).

    python paper_2006_12608_amd/build.py

Run as a script (or loaded by file path): importing the package itself loads
the library, which must not be needed to rebuild it.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libsj.so")
BUILD_DIR = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["sj_api.cpp", "sj_aux.hip", "sj_join_f16.hip", "sj_join_bf16.hip", "sj_join_i8.hip",
           "sj_lsh_api.cpp", "sj_lsh.hip", "sj_jl_api.cpp", "sj_jl.hip"]
PEAK_SOURCE = os.path.join("peak", "mfma_peak.hip")
PEAK_OUT = os.path.join(HERE, "libsj_peak.so")
# Packed-fp32 instructions are kept out of the generated code (they are not
# needed here and some of their forms are unreliable on this hardware).
# MFMA results stay in arch VGPRs so the fused epilogue reads them directly.
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(os.path.basename(src))[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd.insert(1, "-xhip")
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{r.stderr}")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp%d" % os.getpid()
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking {os.path.basename(out)} failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Compile every source and link libsj.so (the join) and libsj_peak.so (the
    MFMA-only throughput probe bench.py reports beside the spec peak); returns
    the path of libsj.so."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES) + 1, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES + [PEAK_SOURCE]))
    _link(objs[:-1], OUT)
    _link(objs[-1:], PEAK_OUT)
    if verbose:
        print(f"built {OUT} and {PEAK_OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
