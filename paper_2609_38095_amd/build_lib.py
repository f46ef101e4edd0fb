"""Compile libzo.so for gfx950 in-tree (hipcc for the HIP sweep, the host compiler for the rest),
and libzo_calib.so, the read-modify-write ceiling probe the benchmark measures beside it (the
sweeps' streaming loop with the probe work replaced by an XOR)."""

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libzo.so")
CALIB_SRC = os.path.join(PKG, "calib", "rmw_ceiling.hip")
CALIB_LIB = os.path.join(PKG, "libzo_calib.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# -packed-fp32-ops off: no v_pk_{add,mul,fma}_f32 in the device code.
DEVICE_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-fast-math"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose=False):
    """Compile every source and link libzo.so; always recompiles. Returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        raise RuntimeError("no host C++ compiler found")
    objs = []
    for name in sorted(os.listdir(CSRC)):
        src = os.path.join(CSRC, name)
        obj = os.path.join(BUILD, name + ".o")
        if name.endswith(".hip"):
            _run([HIPCC, *DEVICE_FLAGS, "-I", INCLUDE, "-c", src, "-o", obj], verbose)
        elif name.endswith(".cpp"):
            _run([cxx, *HOST_FLAGS, "-I", INCLUDE, "-c", src, "-o", obj], verbose)
        else:
            continue
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    # the ceiling kernel runs the sweeps' streaming loop (csrc/zo_stream.h) under their launch
    # plan (the host planner's object, linked in)
    calib_obj = os.path.join(BUILD, "rmw_ceiling.hip.o")
    _run([HIPCC, *DEVICE_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", CALIB_SRC, "-o", calib_obj], verbose)
    tmp = CALIB_LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, calib_obj,
          os.path.join(BUILD, "zo_plan.cpp.o")], verbose)
    os.replace(tmp, CALIB_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
