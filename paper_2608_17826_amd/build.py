"""Build the BSR HIP library (libbsr.so) for gfx950 in-tree.

Every source is compiled with hipcc for gfx950 with packed-FP32 disabled,
then linked into ``paper_2608_17826_amd/libbsr.so`` next to this file.
Run ``python -m paper_2608_17826_amd.build`` or call :func:`build`.
"""

from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbsr.so")

SOURCES = ["bsr_kernels.hip", "bsr_runtime.cpp", "bsr_file_tier.cpp"]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("build step failed: " + " ".join(cmd))
    return r


C_CONSUMER_SRC = os.path.join(ROOT, "tests", "c_abi", "gpu_restore.cpp")
C_CONSUMER = os.path.join(ROOT, "tests", "c_abi", "gpu_restore")


def build_c_consumer(verbose: bool = False) -> str:
    """The torch-free test consumer of the C ABI, linked against libbsr.so
    (found next to the package via a relative rpath)."""
    tmp = C_CONSUMER + ".tmp"
    _run([HIPCC, "-O2", "-std=c++17", f"-I{INCLUDE}", C_CONSUMER_SRC, f"-L{PKG}", "-lbsr",
          "-Wl,-rpath,$ORIGIN/../../paper_2608_17826_amd", "-o", tmp])
    os.replace(tmp, C_CONSUMER)
    if verbose:
        print("built", C_CONSUMER)
    return C_CONSUMER


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        # a fixed compilation-unit id keeps the device code object independent
        # of where the tree is built (it is otherwise derived from the path)
        lang = ["-x", "hip", "-cuid=" + os.path.splitext(src)[0]] if src.endswith(".hip") else []
        _run([HIPCC, *FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, "-lpthread"])
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    build_c_consumer(verbose)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
