"""Builds liblighthouse.so (HIP kernels + C ABI) and the measurement probe libceiling.so for gfx950
with hipcc, in-tree."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "liblighthouse.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["api.cpp", "k_pool_score.hip", "k_select.hip", "k_gather_scatter.hip", "k_sdpa.hip", "k_sdpa_mfma.hip"]
# measurement probe, a library of its own (not part of the attention path)
CEILING_SOURCE = "k_ceiling.hip"
CEILING_OUT = os.path.join(HERE, "libceiling.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         # never emit packed fp32 ALU ops (v_pk_*_f32)
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def _link(objs, out):
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES) + 1)) as ex:
        objs = list(ex.map(_compile, SOURCES + [CEILING_SOURCE]))
    _link(objs[:-1], OUT)
    _link(objs[-1:], CEILING_OUT)
    if verbose:
        print("built", OUT, "and", CEILING_OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
