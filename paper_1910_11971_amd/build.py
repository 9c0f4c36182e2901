"""Build the HIP library ``libcci.so`` for gfx950 (in-tree, next to this file).

    python -m paper_1910_11971_amd.build

Every kernel source is compiled with hipcc for gfx950 only, with packed-FP32
instruction selection disabled (-packed-fp32-ops), then linked with the host
C ABI layer into one shared library that exports the functions declared in
include/cci.h.
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
OUT = os.path.join(HERE, "libcci.so")
BUILD_DIR = os.path.join(ROOT, "_build")

SOURCES = ["cci_api.cpp", "cci_pack.hip", "cci_sparse_mac.hip", "cci_dense_tile.hip", "cci_wide_tile.hip", "cci_narrow.hip",
           "cci_resident.hip", "cci_tap_tile.hip", "cci_stream_tile.hip", "cci_split_k.hip", "cci_glue.hip", "cci_bbs.hip", "cci_train.hip", "cci_grad.hip", "cci_bits.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include"),
]


# Per-source extra flags.  The sparse-MAC kernel branches on wave-uniform
# indices; letting the structurizer leave uniform regions alone keeps those
# branches as plain scalar jumps instead of register-shuffling flow blocks.
EXTRA = {"cci_sparse_mac.hip": ["-mllvm", "-structurizecfg-skip-uniform-regions=true"]}


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = [HIPCC, *COMMON, *EXTRA.get(src, []), *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if verbose and warn.strip():
        print(warn)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = min(len(SOURCES), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    return OUT


def clean() -> None:
    shutil.rmtree(BUILD_DIR, ignore_errors=True)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
