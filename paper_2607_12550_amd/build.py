"""Build ``libjolt.so`` (the C-ABI library) in-tree with hipcc for gfx950.

Usage: ``python -m paper_2607_12550_amd.build`` (or ``build()`` from Python).
Every HIP source is compiled for gfx950 only; host-only sources are compiled
without floating-point contraction so the allocator's double arithmetic is
plain IEEE.  Objects go to ``_build/`` next to this file.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libjolt.so")
BUILD = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

DEVICE_SOURCES = ["k_residual.hip", "k_gemm.hip", "k_gemm16.hip", "k_gram.hip", "k_eig.hip", "k_sytrd.hip", "k_sb.hip", "k_serialize.hip", "k_flash.hip", "k_attend.hip", "k_fused.hip"]
HOST_SOURCES = ["api.cpp", "pipeline.cpp", "diag.cpp"]
STRICT_FP_SOURCES = ["alloc.cpp"]

COMMON = ["-std=c++17", "-O3", "-fPIC", "--offload-arch=gfx950", "-Wall", "-Wno-unused-function",
          "-Wno-unused-variable", "-Wno-unused-but-set-variable"]
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str, extra: list[str]) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msg}")
    if msg.strip():
        print(msg, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = [(s, DEVICE_FLAGS) for s in DEVICE_SOURCES] + [(s, []) for s in HOST_SOURCES] + \
           [(s, ["-ffp-contract=off"]) for s in STRICT_FP_SOURCES]
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        objs = list(ex.map(lambda j: _compile(*j), jobs))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
