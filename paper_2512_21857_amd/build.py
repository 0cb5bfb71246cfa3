"""Builds libadt.so (the HIP kernels and the C ABI) in-tree with hipcc for gfx950, and
libadt_debug.so, the same sources with the device invariant checks compiled in
(ADT_DEVICE_CHECKS=1).

Usage: python -m paper_2512_21857_amd.build   (or build() from Python)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libadt.so")
OUT_DEBUG = os.path.join(PKG, "libadt_debug.so")
BUILD_DIR = os.path.join(PKG, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = [
    "api.hip",
    "kernels/attn.hip",
    "kernels/gemm.hip",
    "kernels/gemm_nt.hip",
    "kernels/rows.hip",
    "kernels/select.hip",
    "kernels/small.hip",
    "kernels/accept_sample.hip",
    "kernels/knn.hip",
    "kernels/probe.hip",
]

# Packed fp32 VALU instructions are disabled for the device code.
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]


def _compile(job) -> str:
    src, debug = job
    obj = os.path.join(BUILD_DIR, ("debug_" if debug else "") + src.replace("/", "_").replace(".hip", ".o"))
    cmd = [HIPCC, *FLAGS, *(["-DADT_DEVICE_CHECKS=1"] if debug else []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    warn = [l for l in r.stderr.splitlines() if "warning" in l and "packed-fp32-ops" not in l]
    if warn:
        sys.stderr.write("\n".join(warn) + "\n")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = [(s, False) for s in SOURCES] + [(s, True) for s in SOURCES]
    with ThreadPoolExecutor(min(8, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, jobs))
    _link(objs[:len(SOURCES)], OUT)
    _link(objs[len(SOURCES):], OUT_DEBUG)
    if verbose:
        print("built", OUT, "and", OUT_DEBUG)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
