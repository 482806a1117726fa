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
           "sj_lsh_api.cpp", "sj_lsh.hip", "sj_jl_api.cpp", "sj_jl.hip", "sj_front.hip", "sj_sort.hip"]
PEAK_SOURCE = os.path.join("peak", "mfma_peak.hip")
PEAK_OUT = os.path.join(HERE, "libsj_peak.so")
# Packed-fp32 instructions are kept out of the generated code (they are not
# needed here and some of their forms are unreliable on this hardware).
# MFMA results stay in arch VGPRs so the fused epilogue reads them directly.
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _obj(src: str) -> str:
    return os.path.join(BUILD_DIR, os.path.splitext(os.path.basename(src))[0] + ".o")


def _deps(path: str, seen=None) -> set:
    """The file and every local header it includes (recursively)."""
    import re
    seen = set() if seen is None else seen
    if path in seen or not os.path.exists(path):
        return seen
    seen.add(path)
    for inc in re.findall(r'^\s*#include\s+"([^"]+)"', open(path).read(), flags=re.M):
        for d in (os.path.dirname(path), CSRC, os.path.join(ROOT, "include")):
            cand = os.path.join(d, inc)
            if os.path.exists(cand):
                _deps(cand, seen)
                break
    return seen


def _stale(src: str) -> bool:
    obj = _obj(src)
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    return any(os.path.getmtime(f) > t for f in _deps(os.path.join(CSRC, src)))


def _compile(src: str) -> str:
    obj = _obj(src)
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


def build(verbose: bool = False, only_stale: bool = False) -> str:
    """Compile every source (only_stale: only those whose object is older than
    the source or a header it includes) and link libsj.so (the join) and
    libsj_peak.so (the MFMA-only loop bench.py --mfma-loop runs); returns the
    path of libsj.so."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = SOURCES + [PEAK_SOURCE]
    todo = [s for s in srcs if _stale(s)] if only_stale else srcs
    with ThreadPoolExecutor(max_workers=min(len(srcs), os.cpu_count() or 4)) as ex:
        list(ex.map(_compile, todo))
    objs = [_obj(s) for s in srcs]
    _link(objs[:-1], OUT)
    _link(objs[-1:], PEAK_OUT)
    if verbose:
        print(f"built {OUT} and {PEAK_OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True, only_stale="--changed" in sys.argv[1:])
    sys.exit(0)
