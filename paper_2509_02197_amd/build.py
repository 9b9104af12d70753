"""Build step for libadst.so (gfx950).

Host sources are compiled as C++ and the kernels as HIP, all with hipcc,
then linked into ``libadst.so`` inside the package directory. Every compile
uses -ffp-contract=off (the forward steps are bit-reproducible in the
documented evaluation order) and disables packed-fp32 instructions.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libadst.so")
ARCH = "gfx950"
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HOST_SOURCES = ["planner.cpp", "ilp.cpp", "abi.cpp"]
HIP_SOURCES = ["kernels.hip", "allencahn.hip", "jacobi_march.hip", "gauss_seidel.hip",
               "static_ws.hip"]

COMMON = ["-std=c++17", "-O3", "-fPIC", "-ffp-contract=off", "-Wall",
          "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
DEVICE = ["--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc():
    for c in ("/opt/rocm/bin/hipcc", "hipcc"):
        if os.path.isabs(c) and os.path.exists(c):
            return c
    return "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("compile failed: " + " ".join(cmd))
    return r


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    jobs = []
    for s in HOST_SOURCES:
        jobs.append([hipcc, "-x", "c++", "-D__HIP_PLATFORM_AMD__=1",
                     "-I" + os.path.join(ROCM, "include")] + COMMON +
                    ["-c", os.path.join(CSRC, s), "-o", os.path.join(BUILD, s + ".o")])
    for s in HIP_SOURCES:
        jobs.append([hipcc, "-x", "hip"] + COMMON + DEVICE +
                    ["-c", os.path.join(CSRC, s), "-o", os.path.join(BUILD, s + ".o")])
    with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    objs = [os.path.join(BUILD, s + ".o") for s in HOST_SOURCES + HIP_SOURCES]
    _run([hipcc, "-shared", "--offload-arch=" + ARCH, "-o", LIB + ".tmp"] + objs +
         ["-L" + os.path.join(ROCM, "lib"), "-lrocprofiler-sdk-roctx",
          "-Wl,-rpath," + os.path.join(ROCM, "lib")], verbose)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
