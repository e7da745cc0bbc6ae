"""Build libmma.so in-tree for gfx950 with hipcc.

Usage: python paper_2512_16056_amd/build.py   (or __graft_entry__.build()).
The library is placed next to this file so that it travels with the source tree.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(ROOT, "_build", "obj")
LIB = os.path.join(HERE, "libmma.so")
NATIVE_LIB = os.path.join(HERE, "libmma_native.so")  # hipMemcpyAsync comparators for the benchmark
INTERPOSE_LIB = os.path.join(HERE, "libmma_interpose.so")  # LD_PRELOAD: hipMemcpy* -> libmma
NATIVE_BATCH = os.path.join(HERE, "native_batch")  # hipMemcpyBatchAsync comparator (its own process)
CXX = os.environ.get("CXX", "g++")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result", f"-I{os.path.join(ROOT, 'include')}"]
# Device code: gfx950 only; no packed-FP32 instruction selection.
DEVICE = [f"--offload-arch={ARCH}", "-x", "hip", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
SOURCES = {
    "mma_kernels.hip": DEVICE,
    "mma_runtime.cpp": ["-x", "c++", "-D__HIP_PLATFORM_AMD__", f"-I{os.path.join(ROCM, 'include')}"],
    "mma_plan.cpp": ["-x", "c++"],
}


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose: bool = False) -> str:
    """Compile every source and link libmma.so; returns the library path."""
    os.makedirs(OBJ, exist_ok=True)
    jobs = []
    for src, extra in SOURCES.items():
        obj = os.path.join(OBJ, src + ".o")
        cmd = [HIPCC, *extra, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
        jobs.append((cmd, obj))
    with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        for r in ex.map(lambda j: _run(j[0]), jobs):
            if verbose and (r.stdout or r.stderr):
                print(r.stdout, r.stderr, file=sys.stderr)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *[o for _, o in jobs], "-o", tmp,
          f"-L{os.path.join(ROCM, 'lib')}", "-lhsa-runtime64", "-lpthread"])
    os.replace(tmp, LIB)
    tmp = NATIVE_LIB + ".tmp"
    nobj = [os.path.join(OBJ, "native_baseline.cpp.o"), os.path.join(OBJ, "native_probes.hip.o")]
    _run([HIPCC, "-x", "c++", "-D__HIP_PLATFORM_AMD__", f"-I{os.path.join(ROCM, 'include')}", *COMMON, "-c",
          os.path.join(CSRC, "native_baseline.cpp"), "-o", nobj[0]])
    _run([HIPCC, *DEVICE, *COMMON, "-c", os.path.join(CSRC, "native_probes.hip"), "-o", nobj[1]])
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *nobj, "-o", tmp, f"-L{os.path.join(ROCM, 'lib')}",
          "-lamdhip64", "-lhsa-runtime64", "-ldl"])
    os.replace(tmp, NATIVE_LIB)
    # LD_PRELOAD interposer: host C++ only, linked against neither the HIP runtime nor libmma.so
    # (both are resolved at run time inside the process).
    tmp = INTERPOSE_LIB + ".tmp"
    _run([CXX, "-std=c++17", "-O2", "-fPIC", "-shared", "-Wall", "-D__HIP_PLATFORM_AMD__",
          f"-I{os.path.join(ROCM, 'include')}", f"-I{os.path.join(ROOT, 'include')}",
          os.path.join(CSRC, "mma_interpose.cpp"), "-o", tmp, "-ldl"])
    os.replace(tmp, INTERPOSE_LIB)
    # The batched comparator links the system ROCm runtime (the one torch bundles does not export
    # hipMemcpyBatchAsync); DT_RPATH, so that no LD_LIBRARY_PATH entry can swap it for another.
    tmp = NATIVE_BATCH + ".tmp"
    _run([CXX, "-std=c++17", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__", f"-I{os.path.join(ROCM, 'include')}",
          os.path.join(CSRC, "native_batch.cpp"), "-o", tmp, f"-L{os.path.join(ROCM, 'lib')}", "-lamdhip64",
          f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-Wl,--disable-new-dtags"])
    os.replace(tmp, NATIVE_BATCH)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
