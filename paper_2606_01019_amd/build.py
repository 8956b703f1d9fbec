"""Build libhvd.so (HIP, gfx950) and libhvd_host.so (host-only state machine).

Usage: python -m paper_2606_01019_amd.build   (or build() from Python).
Outputs go next to this file; object files go to _build/.
"""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(os.path.dirname(PKG), "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhvd.so")
HOST_LIB = os.path.join(PKG, "libhvd_host.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# hipcc is told not to form packed fp32 instructions on its own.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", "-Wall", "-Wno-unused-function"]

HIP_SOURCES = ["gemm.hip", "gemm_tiled.hip", "attn.hip", "attn_o.hip", "misc.hip", "scratch.hip", "flow.hip", "peak.hip"]
HOST_SOURCES = ["api.cpp", "host_state.cpp"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "not a recognized feature" not in l
                    and "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        jobs.append([HIPCC, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, "-c",
                     os.path.join(CSRC, src), "-o", obj])
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        jobs.append([HIPCC, f"--offload-arch={ARCH}", *COMMON, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as pool:
        outs = list(pool.map(_run, jobs))
    objs = [j[-1] for j in jobs]
    tmp = LIB + ".tmp"
    outs.append(_run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]))
    os.replace(tmp, LIB)
    # host-only library for CPU tests of the page allocator / state machine
    tmp = HOST_LIB + ".tmp"
    outs.append(_run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared",
                      os.path.join(CSRC, "host_state.cpp"), os.path.join(CSRC, "host_capi.cpp"), "-o", tmp]))
    os.replace(tmp, HOST_LIB)
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
