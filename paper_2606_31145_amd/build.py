"""Build libsekv.so in-tree with hipcc for gfx950."""

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG, "libsekv.so")
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Device code: no packed-fp32 instructions (their use is disabled on this target).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", f"-I{INCLUDE}", f"-I{CSRC}"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")


def build(verbose: bool = False) -> str:
    """Compile the kernels and the host layer and link libsekv.so; returns its path."""
    bdir = os.path.join(PKG, "_build")
    os.makedirs(bdir, exist_ok=True)
    k_obj = os.path.join(bdir, "sekv_kernels.o")
    t_obj = os.path.join(bdir, "sekv_tier.o")
    a_obj = os.path.join(bdir, "sekv_api.o")
    for src, obj in (("sekv_kernels.hip", k_obj), ("sekv_tier.hip", t_obj)):
        _run([HIPCC, *COMMON, f"--offload-arch={ARCH}", *DEVICE_FLAGS, "-c",
              os.path.join(CSRC, src), "-o", obj], verbose)
    _run([HIPCC, *COMMON, f"--offload-arch={ARCH}", "-c", os.path.join(CSRC, "sekv_api.cpp"), "-o", a_obj],
         verbose)
    tmp = LIB_PATH + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", k_obj, t_obj, a_obj, "-o", tmp], verbose)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
