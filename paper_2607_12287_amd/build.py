"""Build libincvit.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_12287_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libincvit.so")
DRIVE = os.path.join(HERE, "incvit_drive")
SOURCES = ["incvit_api.hip", "k_embed.hip", "k_select.hip", "k_gemm.hip", "k_gemm_qkv.hip",
           "k_gemm_fc1.hip", "k_gemm_part.hip", "k_gemm_res.hip", "k_gemm_att.hip", "k_gemm_down.hip", "k_gemm_tiled.hip", "k_rows.hip", "k_attn.hip", "k_misc.hip", "k_flow.hip"]
# the fixed-order fp32 embedding and cosine must not be contracted beyond the
# explicit fma intrinsics
NO_CONTRACT = {"k_embed.hip"}

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["--offload-arch=" + ARCH, "-O3", "-fPIC", "-std=c++17",
          # packed fp32 ops are kept out of the generated code
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    flags = list(COMMON)
    if src in NO_CONTRACT:
        flags.append("-ffp-contract=off")
    cmd = [HIPCC, *flags, "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stderr}")
    return obj


def objects(sources=SOURCES) -> list:
    """Object files of the given sources, compiling only those older than their
    source or any header (the sanitizer test links its own library from them
    and leaves libincvit.so as it is)."""
    os.makedirs(BUILD, exist_ok=True)
    headers = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hpp")]
    headers += [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))]
    newest = max(os.path.getmtime(h) for h in headers)

    def obj(src):
        return os.path.join(BUILD, os.path.splitext(src)[0] + ".o")

    def fresh(src):
        o = obj(src)
        return os.path.exists(o) and os.path.getmtime(o) >= max(newest, os.path.getmtime(os.path.join(CSRC, src)))

    stale = [src for src in sources if not fresh(src)]
    if stale:
        with cf.ThreadPoolExecutor(max_workers=min(10, os.cpu_count() or 1)) as ex:
            list(ex.map(_compile, stale))
    return [obj(src) for src in sources]


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libincvit.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(10, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    # the native driver (counter passes run it without a Python runtime)
    tmp = DRIVE + f".tmp{os.getpid()}"
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-O2", "-std=c++17", "-x", "hip", os.path.join(CSRC, "incvit_drive.cpp"),
           "-I", os.path.join(ROOT, "include"), "-L", HERE, "-lincvit", "-Wl,-rpath,$ORIGIN", "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"driver build failed:\n{res.stderr}")
    os.replace(tmp, DRIVE)
    if verbose:
        print("built", LIB, "and", DRIVE)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
