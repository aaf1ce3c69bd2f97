"""Builds libmoa.so (HIP kernels for gfx950 + the C-ABI host code) in-tree.

Usage: python -m paper_2406_14909_amd.build
Cross-compiles without a GPU; the library lands next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from typing import List

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG_DIR, "_build")
LIB_PATH = os.path.join(PKG_DIR, "libmoa.so")
# Measurement helpers (not part of the library): the streaming-read and
# matrix-core ceilings of the GPU.
PROBES = ["stream_read", "mfma_loop"]

HIP_SOURCES = ["kv_append.hip", "decode.hip", "prefill.hip", "influence.hip", "rule_loss.hip"]
HOST_SOURCES = ["moa_api.cpp"]

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX", "g++")

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-mcode-object-version=5",
    # packed fp32 VALU forms are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]
HOST_FLAGS = ["-std=c++17", "-O2", "-fPIC", "-ffp-contract=off", "-Wall", "-Wextra",
              "-D__HIP_PLATFORM_AMD__"]


def _run_all(cmds: List[List[str]]) -> None:
    procs = [(c, subprocess.Popen(c, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)) for c in cmds]
    failed = []
    for c, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        if p.returncode != 0:
            failed.append((c, text))
        elif "warning" in text:
            sys.stderr.write(text)
    if failed:
        msg = "\n\n".join(" ".join(c) + "\n" + t for c, t in failed)
        raise RuntimeError("libmoa build failed:\n" + msg)


def build(verbose: bool = False) -> str:
    """Compiles every source and links libmoa.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    includes = [f"-I{INCLUDE}", f"-I{CSRC}"]
    objs, cmds = [], []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        cmds.append([HIPCC, *HIP_FLAGS, *includes, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        cmds.append([CXX, *HOST_FLAGS, *includes, "-I/opt/rocm/include", "-c",
                     os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    if verbose:
        for c in cmds:
            print(" ".join(c))
    _run_all(cmds)
    tmp = LIB_PATH + ".tmp"
    _run_all([[HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]] +
             [[HIPCC, *HIP_FLAGS, os.path.join(PKG_DIR, "calibration", p + ".hip"), "-o", os.path.join(BUILD_DIR, p)]
              for p in PROBES])
    shutil.move(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
