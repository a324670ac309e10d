"""Build libdendsn.so (HIP, gfx950) in-tree with hipcc.

Each translation unit compiles in its own hipcc process, in parallel, into
``_build/``; the objects are then linked into ``libdendsn.so`` next to this file.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdendsn.so")

# (source, extra flags, object name).  The backward units compile once per
# surrogate derivative (-DDENDSN_SG=0: atan, 1: sigmoid); the heaviest first.
_BWD = ["dendsn_bwd_bf16.hip", "dendsn_bwd_bf16_kc.hip", "dendsn_bwd_f32.hip", "dendsn_bwd_f32_kc.hip",
        "dendsn_bwd_f32_cm.hip", "dendsn_bwd_bf16_cm.hip"]
_OTHER = ["dendsn_fwd_f32_cm.hip", "dendsn_fwd_bf16_cm.hip", "dendsn_fwd_f32_kc.hip", "dendsn_fwd_bf16_kc.hip",
          "dendsn_api.hip", "dendsn_fwd_f32.hip", "dendsn_fwd_bf16.hip"]
SOURCES = [(src, [f"-DDENDSN_SG={k}"], f"{src[:-4]}_sg{k}.o") for src in _BWD for k in (0, 1)] + \
          [(src, [], f"{src[:-4]}.o") for src in _OTHER]

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

# -ffp-contract=off: the forward kernel and the backward's recompute must round
# every operation the same way; fused multiply-adds are written out as fmaf.
# Packed FP32 instructions are disabled.
CFLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(unit) -> str:
    src, extra, name = unit
    obj = os.path.join(BUILD, name)
    cmd = [HIPCC, *CFLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True, jobs: int | None = None) -> str:
    """Compile every HIP source for gfx950 and link libdendsn.so. Returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
