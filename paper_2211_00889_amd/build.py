"""Builds libnbsgd.so (host C++ + gfx950 HIP kernels) and the synthetic-input
fill library in-tree.  ``python -m paper_2211_00889_amd.build``."""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJ = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libnbsgd.so")
SYNTH_LIB = os.path.join(ROOT, "synth", "libsynth.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# gfx950 device code: no packed-fp32 instructions (issued by the compiler from
# plain float code otherwise), full optimisation.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wno-unused-command-line-argument"]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wall", "-Wextra"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")
    return r


def _atomic_link(cmd_prefix, out, verbose):
    tmp = out + ".tmp"
    _run(cmd_prefix + ["-o", tmp], verbose)
    os.replace(tmp, out)


def build(verbose: bool = False) -> None:
    os.makedirs(OBJ, exist_ok=True)
    cxx = shutil.which("g++") or "g++"
    host_o = os.path.join(OBJ, "host.o")
    _run([cxx, *CXX_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "host.cpp"),
          "-o", host_o], verbose)
    matcha_o = os.path.join(OBJ, "matcha.o")
    _run([cxx, *CXX_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "matcha.cpp"),
          "-o", matcha_o], verbose)
    step_o = os.path.join(OBJ, "step.o")
    _run([HIPCC, *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "step.hip"),
          "-o", step_o], verbose)
    mlp_o = os.path.join(OBJ, "mlp.o")
    _run([HIPCC, *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "mlp.hip"),
          "-o", mlp_o], verbose)
    _atomic_link([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", host_o, matcha_o, step_o, mlp_o],
                 LIB, verbose)
    _atomic_link([HIPCC, *HIP_FLAGS, "-shared", os.path.join(ROOT, "synth", "fill.hip")],
                 SYNTH_LIB, verbose)


if __name__ == "__main__":
    build(verbose=True)
    print("built", LIB, SYNTH_LIB)
