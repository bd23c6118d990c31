"""Compile the gfx950 HIP library libinfllm.so in-tree (hipcc, no JIT cache).

    python -m paper_2402_04617_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libinfllm.so")
PEAKS = os.path.join(PKG, "infllm_peaks")
TOPK_CMP = os.path.join(PKG, "infllm_topk_compare")

SOURCES = ["abi.cpp", "append.hip", "build_units.hip", "score.hip", "topk.hip", "attend_mfma.hip",
           "attend.hip", "attend_decode.hip", "merge.hip", "mass.hip"]

# Packed fp32 ops are disabled for all device code (the host pass warns that it
# does not know the feature; that is harmless).
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def build(verbose: bool = False, jobs: int = 8) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)

    def compile_one(src: str) -> str:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                        if "packed-fp32-ops" not in l and l.strip())
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
        if verbose and msg:
            print(msg, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max(1, jobs)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    # the measured-peak probe that bench.py runs next to the library (a separate program)
    cmd = [hipcc, *FLAGS, os.path.join(PKG, "probes", "peaks.hip"), "-o", PEAKS + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on probes/peaks.hip:\n" + r.stdout + r.stderr)
    os.replace(PEAKS + ".tmp", PEAKS)
    # radix select against a bitonic top-k on the lookup's row shapes (a separate program)
    cmd = [hipcc, *FLAGS, os.path.join(PKG, "probes", "topk_compare.hip"), "-ldl", "-o", TOPK_CMP + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on probes/topk_compare.hip:\n" + r.stdout + r.stderr)
    os.replace(TOPK_CMP + ".tmp", TOPK_CMP)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
