"""Build the gfx950 shared library ``librwttt.so`` in-tree with hipcc.

Usage: ``python -m paper_2605_28053_amd.build`` (or ``build()`` from Python).
The library holds the host planner/owner table and the HIP kernels behind the
C ABI declared in ``include/rwttt.h``.
"""

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "librwttt.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed fp32 instructions are disabled for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed: " + " ".join(cmd))
    # the host pass does not know the device-only feature flag; drop that noise
    noise = "'-packed-fp32-ops' is not a recognized feature"
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if out.strip():
        sys.stderr.write(out + "\n")


def build(verbose=False):
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    k_obj = os.path.join(objdir, "rwttt_kernels.o")
    d_obj = os.path.join(objdir, "rwttt_adapter.o")
    a_obj = os.path.join(objdir, "rwttt_api.o")
    _run([HIPCC, "-c", f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS,
          os.path.join(CSRC, "rwttt_kernels.hip"), "-o", k_obj])
    _run([HIPCC, "-c", f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS,
          os.path.join(CSRC, "rwttt_adapter.hip"), "-o", d_obj])
    _run([HIPCC, "-c", f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS,
          os.path.join(CSRC, "rwttt_api.cpp"), "-o", a_obj])
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", f"--offload-arch={ARCH}", "-fPIC", a_obj, k_obj, d_obj, "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
