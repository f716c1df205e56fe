"""Build libsekv.so (and its phase-trace variant libsekv_trace.so) in-tree with hipcc for gfx950.

The step kernel's sixteen instantiations are split over four translation units (storage
type x head_dim) so that they compile in parallel.  The trace variant is the same source
compiled with SEKV_PHASE_TRACE: its kernels stamp per-item phase times into a buffer the
caller attaches with sekv_phase_trace (a diagnostic build; the product path loads
libsekv.so).
"""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG, "libsekv.so")
TRACE_LIB_PATH = os.path.join(PKG, "libsekv_trace.so")
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Device code: no packed-fp32 instructions (their use is disabled on this target).
# Device code must not use scratch memory (a build whose kernel spilled registers to scratch
# gave wrong results): any kernel with a stack frame fails to compile.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-Xarch_device", "-Wframe-larger-than=0", "-Xarch_device", "-Werror=frame-larger-than"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", f"-I{INCLUDE}", f"-I{CSRC}"]
INSTANCES = [("BF16", 128), ("BF16", 64), ("F32", 128), ("F32", 64)]

# every source the kernels are built from (the bench hashes these to tie counter
# figures to the kernel code they were taken on)
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in
                  ("sekv_internal.h", "sekv_step.h", "sekv_step_inst.hip", "sekv_kernels.hip")]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")


def _jobs(bdir, trace):
    """(command, object) pairs of one library variant."""
    tflag = ["-DSEKV_PHASE_TRACE"] if trace else []
    sfx = "_trace" if trace else ""
    jobs = []
    for t, d in INSTANCES:
        obj = os.path.join(bdir, f"sekv_step_{t}_{d}{sfx}.o")
        jobs.append(([HIPCC, *COMMON, f"--offload-arch={ARCH}", *DEVICE_FLAGS, *tflag,
                      f"-DSEKV_T={t}", f"-DSEKV_D={d}", "-c",
                      os.path.join(CSRC, "sekv_step_inst.hip"), "-o", obj], obj))
    for src in ("sekv_kernels.hip", "sekv_tier.hip", "sekv_noalloc.hip", "sekv_gate.hip"):
        obj = os.path.join(bdir, src.replace(".hip", ".o"))
        jobs.append(([HIPCC, *COMMON, f"--offload-arch={ARCH}", *DEVICE_FLAGS, "-c",
                      os.path.join(CSRC, src), "-o", obj], obj))
    obj = os.path.join(bdir, f"sekv_build{sfx}.o")        # the builder's SVD has phase marks too
    jobs.append(([HIPCC, *COMMON, f"--offload-arch={ARCH}", *DEVICE_FLAGS, *tflag, "-c",
                  os.path.join(CSRC, "sekv_build.hip"), "-o", obj], obj))
    obj = os.path.join(bdir, f"sekv_api{sfx}.o")
    jobs.append(([HIPCC, *COMMON, f"--offload-arch={ARCH}", *tflag, "-c",
                  os.path.join(CSRC, "sekv_api.cpp"), "-o", obj], obj))
    obj = os.path.join(bdir, "sekv_build_api.o")
    jobs.append(([HIPCC, *COMMON, f"--offload-arch={ARCH}", "-c",
                  os.path.join(CSRC, "sekv_build_api.cpp"), "-o", obj], obj))
    obj = os.path.join(bdir, "sekv_host.o")
    jobs.append(([HIPCC, *COMMON, "-c", os.path.join(CSRC, "sekv_host.cpp"), "-o", obj], obj))
    return jobs


def build(verbose: bool = False, trace: bool = True) -> str:
    """Compile and link libsekv.so (and libsekv_trace.so unless trace=False); returns
    the path of libsekv.so."""
    bdir = os.path.join(PKG, "_build")
    os.makedirs(bdir, exist_ok=True)
    variants = [(False, LIB_PATH)] + ([(True, TRACE_LIB_PATH)] if trace else [])
    per = {v: _jobs(bdir, v) for v, _ in variants}
    uniq = {}
    for v, _ in variants:
        for cmd, obj in per[v]:
            uniq[obj] = cmd
    workers = max(1, min(16, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda c: _run(c, verbose), uniq.values()))
    for v, path in variants:
        tmp = path + ".tmp"
        _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *[o for _, o in per[v]],
              "-o", tmp], verbose)
        os.replace(tmp, path)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True, trace="--no-trace" not in sys.argv))
