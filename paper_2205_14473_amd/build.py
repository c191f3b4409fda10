"""Build ``libea.so`` (the HIP kernels + C ABI) in-tree for gfx950.

Flags that matter for results:
  -ffp-contract=off      every a*b+c stays two binary32 roundings (no FMA)
  (no fast-math)         binary32 division and square root are correctly rounded
  -packed-fp32-ops off   no packed FP32 instructions are generated

Each source is compiled in two passes, as the HIP driver does internally: a
device pass for gfx950, which alone gets the target feature that turns packed
FP32 off, and a host pass that embeds the device pass's fat binary.  Both use
one compilation-unit ID (it names file-scope device variables, which the host
registers by name).  The objects are byte-identical to a one-command hipcc
build with the same flags, and the host pass does not see a device feature it
would warn about.
"""
import hashlib
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
CLANG = os.environ.get("HIP_CLANG", "/opt/rocm/lib/llvm/bin/clang++")

FLAGS = [
    "-x", "hip", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]
DEVICE_FLAGS = ["--cuda-device-only", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run_all(cmds, verbose):
    procs = []
    for cmd in cmds:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd)))
    failed = [cmd for cmd, p in procs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])


def build(verbose: bool = False, extra=()) -> str:
    """Compile the library (always): the device passes of all sources in
    parallel, then their host passes, then one link; returns its path."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    dev, host, objs = [], [], []
    for src in SOURCES:
        base = os.path.join(objdir, os.path.basename(src))
        cuid = "-cuid=" + hashlib.sha256(os.path.basename(src).encode()).hexdigest()[:16]
        dev.append([CLANG, *FLAGS, cuid, *extra, *DEVICE_FLAGS, src, "-o", base + ".hipfb"])
        host.append([CLANG, *FLAGS, cuid, *extra, "--cuda-host-only", "-c", "-Xclang", "-fcuda-include-gpubinary",
                     "-Xclang", base + ".hipfb", src, "-o", base + ".o"])
        objs.append(base + ".o")
    _run_all(dev, verbose)
    _run_all(host, verbose)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


# The host code (argument checks, planning, launch set-up) built with
# AddressSanitizer and UndefinedBehaviorSanitizer for the CPU tests; device
# code is unchanged (the last build's device objects are reused).  The
# library is linked without the sanitizer runtime: the process that loads it
# preloads clang's.
SAN_HOST_FLAGS = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
                  "-fno-omit-frame-pointer"]


def build_host_sanitized(outdir: str, verbose: bool = False) -> str:
    """Host passes of every source with SAN_HOST_FLAGS into outdir, then one
    link; needs the device objects of build().  Returns the library's path."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(outdir, exist_ok=True)
    host, objs = [], []
    for src in SOURCES:
        bn = os.path.basename(src)
        fb = os.path.join(objdir, bn + ".hipfb")
        if not os.path.exists(fb):
            raise FileNotFoundError(f"{fb}: run build() first")
        cuid = "-cuid=" + hashlib.sha256(bn.encode()).hexdigest()[:16]
        o = os.path.join(outdir, bn + ".o")
        host.append([CLANG, *FLAGS, cuid, *SAN_HOST_FLAGS, "--cuda-host-only", "-c", "-Xclang",
                     "-fcuda-include-gpubinary", "-Xclang", fb, src, "-o", o])
        objs.append(o)
    _run_all(host, verbose)
    lib = os.path.join(outdir, "libea.so")
    subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", lib], check=True)
    return lib


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True, extra=sys.argv[1:]))
