"""Build libdaso.so (the C-ABI library with its gfx950 kernels) in-tree with hipcc.

Usage: python -m paper_2104_05588_amd.build  (or call build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdaso.so")
CAPI_CLIENT_SRC = os.path.join(ROOT, "tests", "c", "fused_step_capi.c")
CAPI_CLIENT = os.path.join(PKG, "fused_step_capi")  # next to libdaso.so (found through $ORIGIN)
CAPI_CLUSTER_SRC = os.path.join(ROOT, "tests", "c", "daso_cluster_capi.c")
CAPI_CLUSTER = os.path.join(PKG, "daso_cluster_capi")

SOURCES = ["daso_kernels.hip", "daso_api.hip", "daso_host.cpp", "daso_schedule.cpp"]
# The bench's bandwidth-ceiling probes (the step's access pattern without its
# arithmetic): a library of their own, outside the C ABI.
PROBE_SOURCE = "daso_ceiling.hip"
PROBE_LIB = os.path.join(PKG, "libdaso_ceiling.so")

# Numerics flags: binary32 operations must be evaluated exactly as written (no
# contraction into FMA, correctly rounded division, subnormals kept), so the
# kernels reproduce a plain IEEE evaluation bit for bit.  Packed fp32 ALU
# instructions are disabled.
HIP_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-mcode-object-version=5", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: the DASO library needs ROCm's hipcc to build")


def build(verbose: bool = False) -> str:
    """Compile every source into libdaso.so next to this file; returns its path."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    errs = [ln for ln in res.stderr.splitlines() if "warning" in ln and "packed-fp32-ops" not in ln]
    if verbose and errs:
        sys.stderr.write("\n".join(errs) + "\n")
    os.replace(tmp, LIB)
    build_probes(verbose)
    if os.path.exists(CAPI_CLIENT_SRC):
        build_capi_client(verbose)
    return LIB


def build_probes(verbose: bool = False) -> str:
    """libdaso_ceiling.so: the access-pattern probes that bench.py times."""
    tmp = PROBE_LIB + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, os.path.join(CSRC, PROBE_SOURCE), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


def build_capi_client(verbose: bool = False) -> str:
    """The plain C test programs of the ABI (tests/c), linked against libdaso.so."""
    for src, exe in ((CAPI_CLIENT_SRC, CAPI_CLIENT), (CAPI_CLUSTER_SRC, CAPI_CLUSTER)):
        if not os.path.exists(src):
            continue
        cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE, "-I", "/opt/rocm/include",
               src, "-o", exe, "-L", PKG, "-ldaso", "-L", "/opt/rocm/lib", "-lamdhip64",
               "-Wl,-rpath,$ORIGIN", "-Wl,-rpath,/opt/rocm/lib"]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"gcc failed with status {res.returncode}")
    return CAPI_CLIENT


if __name__ == "__main__":
    print(build(verbose=True))
