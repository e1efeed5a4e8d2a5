"""Builds libtetra.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_2609_35465_amd.build   (or build() from Python)
"""

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libtetra.so")

SOURCES = ["tables.cpp", "tetra.hip"]

HIP_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # packed FP32 VALU ops stay off on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core results in ordinary VGPRs: the many-token product scales
    # every block's products on the vector unit, which cannot read AGPRs
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


BUILD_DIR = os.path.join(HERE, "_build")
GEN_SOURCES = ["gen_tables.cpp", "tables.cpp"]


def _run(cmd, verbose, **kw):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"{cmd[0]} failed with status {res.returncode}")
    return res


def generate_tables(verbose: bool = False) -> str:
    """Builds and runs the host table generator; writes the initialisers of
    the device decoder tables to _build/tables_data.inc and returns the
    directory."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    gen = os.path.join(BUILD_DIR, "gen_tables")
    _run([hipcc(), "-O2", "-std=c++17", "-Wno-unused-command-line-argument",
          *[os.path.join(CSRC, s) for s in GEN_SOURCES], "-o", gen], verbose)
    out = _run([gen], verbose).stdout
    path = os.path.join(BUILD_DIR, "tables_data.inc")
    with open(path + ".tmp", "w") as f:
        f.write(out)
    os.replace(path + ".tmp", path)
    return BUILD_DIR


def build(verbose: bool = False) -> str:
    """Compiles every source into libtetra.so next to this file; returns its path."""
    inc = generate_tables(verbose)
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, "-I", inc, *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
