"""Build libhg.so (gfx950) in-tree with hipcc, plus libhg_ceiling.so (the
benchmark's memory-ceiling measurement, not part of the hot path).

Usage: python -m paper_2608_02168_amd.build   (or __graft_entry__.build()).
Always recompiles every source; objects are built in parallel.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libhg.so")
CEILING_LIB = os.path.join(HERE, "libhg_ceiling.so")
ARCH = os.environ.get("HG_OFFLOAD_ARCH", "gfx950")

SOURCES = ["hg_api.hip", "hg_scan.hip", "hg_build.hip", "hg_layer.hip", "hg_hgt.hip", "hg_align.hip", "hg_objective.hip",
           "hg_temporal.hip", "hg_kway.hip"]
CEILING_SOURCES = ["hg_ceiling.hip"]

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str, obj_dir: str) -> str:
    obj = os.path.join(obj_dir, src.replace(".hip", ".o"))
    cmd = [hipcc(), *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link of {os.path.basename(out)} failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = True) -> str:
    obj_dir = os.path.join(HERE, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    srcs = SOURCES + CEILING_SOURCES
    workers = min(len(srcs), max(1, (os.cpu_count() or 2)))
    with cf.ThreadPoolExecutor(workers) as ex:
        objs = dict(zip(srcs, ex.map(lambda s: _compile(s, obj_dir), srcs)))
    _link([objs[s] for s in SOURCES], LIB)
    _link([objs[s] for s in CEILING_SOURCES], CEILING_LIB)
    if verbose:
        print(f"built {LIB}")
        print(f"built {CEILING_LIB}")
    return LIB


if __name__ == "__main__":
    build()
