"""Build libdopr.so (HIP, gfx950) in-tree with hipcc.

Every translation unit is compiled for gfx950 only, with packed-fp32
instruction selection disabled, then linked into one shared library next to
this file.  Run as ``python -m paper_2609_03311_amd._build``.

``python -m paper_2609_03311_amd._build timers`` builds the measurement
library libdopr_timers.so instead: the same sources with the pass kernel's
per-phase cycle counters compiled in (-DDOPR_PASS_TIMERS).  Only
``phase_timing`` loads it.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdopr.so")
TIMERS_BUILD = os.path.join(HERE, "_build", "timers")
TIMERS_LIB = os.path.join(HERE, "libdopr_timers.so")
SOURCES = ["api.hip", "store.hip", "group.hip", "attn.hip", "stream.hip",
           "score.hip", "layer.hip", "salience.hip"]
# per-file flags: the streaming kernel's cursor must stay in scalar
# registers (common-code sinking would move it to scratch memory)
EXTRA = {"stream.hip": ["-mllvm", "-simplifycfg-sink-common=false"]}
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # results must not depend on which template instance or inlining
    # context the compiler fuses multiply-adds in: fuse only where written
    "-ffp-contract=off",
    # no v_pk_{add,mul,fma}_f32 from the compiler's own vectorisation
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found (ROCm is required to build)")
    return path


def _compile(src: str, build_dir: str = BUILD, defs=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *FLAGS, *defs, *EXTRA.get(src, []), "-c",
           os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False, timers: bool = False) -> str:
    build_dir = TIMERS_BUILD if timers else BUILD
    lib = TIMERS_LIB if timers else LIB
    defs = ("-DDOPR_PASS_TIMERS",) if timers else ()
    os.makedirs(build_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, build_dir, defs), SOURCES))
    tmp = lib + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
           *objs, "-lhipblaslt"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(verbose=True, timers=sys.argv[1:] == ["timers"])
    sys.exit(0)
