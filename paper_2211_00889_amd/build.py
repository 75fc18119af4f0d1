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


# The host translation units (plain C++, no HIP): the schedule and mixing
# matrices, MATCHA, the step planner and the MLP shape checks.
HOST_SOURCES = ("host.cpp", "matcha.cpp", "plan.cpp", "mlp_shape.cpp")
# Sanitizers for the host-only test build (g++, no GPU code involved).
SANITIZE_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                  "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False) -> None:
    os.makedirs(OBJ, exist_ok=True)
    cxx = shutil.which("g++") or "g++"
    host_objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(OBJ, src.replace(".cpp", ".o"))
        _run([cxx, *CXX_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj],
             verbose)
        host_objs.append(obj)
    step_o = os.path.join(OBJ, "step.o")
    _run([HIPCC, *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "step.hip"),
          "-o", step_o], verbose)
    mlp_o = os.path.join(OBJ, "mlp.o")
    _run([HIPCC, *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "mlp.hip"),
          "-o", mlp_o], verbose)
    _atomic_link([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *host_objs, step_o, mlp_o],
                 LIB, verbose)
    _atomic_link([HIPCC, *HIP_FLAGS, "-shared", "-I", INCLUDE, os.path.join(ROOT, "synth", "fill.hip")],
                 SYNTH_LIB, verbose)


def build_sanitized_host_tests(out_dir: str, verbose: bool = False):
    """The host translation units and the host-only test programs
    (tests/c/abi_host.c, tests/c/plan_emulation.cpp) built with g++ under
    AddressSanitizer and UndefinedBehaviorSanitizer, linked statically into
    two executables in ``out_dir`` that need no GPU and no HIP runtime.
    Returns their paths."""
    os.makedirs(out_dir, exist_ok=True)
    cxx = shutil.which("g++") or "g++"
    cc = shutil.which("gcc") or "gcc"
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(out_dir, src.replace(".cpp", ".san.o"))
        _run([cxx, *CXX_FLAGS, *SANITIZE_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
              os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    tests_c = os.path.join(ROOT, "tests", "c")
    abi_o = os.path.join(out_dir, "abi_host.san.o")
    _run([cc, "-std=c11", "-Wall", "-Wextra", "-pedantic", "-Werror", *SANITIZE_FLAGS, "-I", INCLUDE,
          "-c", os.path.join(tests_c, "abi_host.c"), "-o", abi_o], verbose)
    abi = os.path.join(out_dir, "abi_host_san")
    _run([cxx, *SANITIZE_FLAGS, abi_o, *objs, "-lm", "-o", abi], verbose)
    emu = os.path.join(out_dir, "plan_emulation_san")
    _run([cxx, "-std=c++17", "-O1", "-Wall", "-Wextra", *SANITIZE_FLAGS, "-I", INCLUDE, "-I", CSRC,
          os.path.join(tests_c, "plan_emulation.cpp"), *objs, "-o", emu], verbose)
    return abi, emu


if __name__ == "__main__":
    build(verbose=True)
    print("built", LIB, SYNTH_LIB)
