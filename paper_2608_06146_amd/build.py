"""Build ``libpadoc_attn.so`` in-tree with hipcc for gfx950.

    python -m paper_2608_06146_amd.build            # incremental
    python -m paper_2608_06146_amd.build --force    # rebuild everything

Objects go to ``_build/`` at the repository root; the shared library is
written next to this file, where the Python binding loads it.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpadoc_attn.so")
ARCH = os.environ.get("PADOC_OFFLOAD_ARCH", "gfx950")

SOURCES = [
    "csrc/host/plan.cpp",
    "csrc/host/session.cpp",
    "csrc/abi.hip",
    "csrc/kernels/tile_mfma_bf16.hip",
    "csrc/kernels/decode_step.hip",
    "csrc/kernels/tile_valu_f32.hip",
    "csrc/kernels/lse_combine.hip",
    "csrc/kernels/bwd.hip",
    "csrc/kernels/append.hip",
    "csrc/kernels/relayout.hip",
]
# Every header under csrc/ (and the public header) enters each object's
# digest, so an edit to any of them rebuilds every object.
HEADERS = sorted(os.path.relpath(os.path.join(d, f), PKG)
                 for d, _, fs in os.walk(os.path.join(PKG, "csrc")) for f in fs if f.endswith((".hpp", ".h")))

# Packed fp32 VALU forms are kept out of device code on purpose: the
# compiler must not form v_pk_{add,mul,fma}_f32 from scalar fp32 code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", os.path.join(ROOT, "include"),
          "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libpadoc_attn)")


def _digest(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    h.update(" ".join(COMMON + DEVICE_FLAGS).encode())
    return h.hexdigest()[:16]


def _compile(cc: str, src: str, force: bool) -> str:
    spath = os.path.join(PKG, src)
    hdrs = [os.path.join(PKG, h) for h in HEADERS] + [os.path.join(ROOT, "include", "padoc_attn.h")]
    tag = _digest([spath] + hdrs)
    obj = os.path.join(BUILD, src.replace("/", "_") + f".{tag}.o")
    if os.path.exists(obj) and not force:
        return obj
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [cc] + COMMON + DEVICE_FLAGS + lang + ["-c", spath, "-o", obj + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(obj + ".tmp", obj)
    return obj


def build(force: bool = True, verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    cc = hipcc()
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(cc, s, force), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--force", action="store_true")
    a = ap.parse_args(argv)
    build(force=a.force, verbose=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
