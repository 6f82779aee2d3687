"""Build libcoco.so for gfx950 with hipcc, in-tree.

Each .hip source is compiled on its own (in parallel) into _build/, then
linked into paper_2607_04181_amd/libcoco.so. Always recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
ROOT = os.path.dirname(PKG)
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libcoco.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 ops are switched off for device code: all fp32 math stays scalar
# VALU. (The host pass prints a harmless "not a recognized feature" note.)
FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-Wall",
         "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         f"-I{os.path.join(ROOT, 'include')}"]
SOURCES = ["rows.hip", "gemm_skinny.hip", "gemm_tile.hip", "gemm_narrow.hip", "attention.hip", "coco_api.hip",
           "probe.hip", "scaling.cpp"]


def build(verbose: bool = False, jobs: int = 8) -> str:
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD, exist_ok=True)
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                            stderr=subprocess.STDOUT, text=True)))
    errors = []
    for src, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            errors.append(f"--- {src} ---\n{out}")
        elif verbose and out.strip():
            print(_filter_notes(out), flush=True)
    if errors:
        raise RuntimeError("HIP compile failed:\n" + "\n".join(errors))
    tmp = LIB + ".tmp"
    # -z defs: an undefined symbol fails the link here, not the first import.
    cmd = [HIPCC, "-shared", "-fPIC", "-Wl,-z,defs", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout)
    shutil.move(tmp, LIB)
    return LIB


def _filter_notes(out: str) -> str:
    return "\n".join(l for l in out.splitlines() if "packed-fp32-ops" not in l)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
