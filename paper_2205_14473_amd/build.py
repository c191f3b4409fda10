"""Build ``libea.so`` (the HIP kernels + C ABI) in-tree for gfx950 with hipcc.

Flags that matter for results:
  -ffp-contract=off      every a*b+c stays two binary32 roundings (no FMA)
  (no fast-math)         binary32 division and square root are correctly rounded
  -packed-fp32-ops off   no packed FP32 instructions are generated
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libea.so")
SOURCES = [os.path.join(CSRC, f) for f in ("ea_kernels.hip", "ea_half_c1.hip", "ea_half_c2.hip", "ea_half_c4.hip",
                                            "ea_half_c8.hip", "ea_sym_c4.hip", "ea_sym_c8.hip", "ea_toy.hip",
                                            "ea_api.cpp")]
HEADERS = [os.path.join(CSRC, f) for f in ("ea_device.hpp", "ea_launch.hpp", "ea_round.hpp")] + \
    [os.path.join(ROOT, "include", "ea.h")]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def build(verbose: bool = False, extra=()) -> str:
    """Compile the library (always): each source to an object, in parallel,
    then one link; returns its path."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for src in SOURCES:
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        jobs.append((cmd, obj, subprocess.Popen(cmd)))
    failed = [cmd for cmd, _, p in jobs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *[o for _, o, _ in jobs], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True, extra=sys.argv[1:]))
