"""Compile the C oracle into ``oracle/liboracle.so`` with gcc.

Test infrastructure only: the product library never links this object.
``-ffp-contract=off`` keeps every a*b+c as two binary32 roundings; no
fast-math flag is used, so division and square root are correctly rounded.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
SOURCES = [os.path.join(HERE, "eao.c")]
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-fno-strict-aliasing", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    """Compile the oracle; returns the path of the shared object."""
    cmd = ["gcc", *CFLAGS, *SOURCES, "-lm", "-o", LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def ensure_built() -> str:
    """Build only when the shared object is missing or older than a source."""
    if os.path.exists(LIB):
        t = os.path.getmtime(LIB)
        srcs = SOURCES + [os.path.join(HERE, "eao.h")]
        if all(os.path.getmtime(s) <= t for s in srcs):
            return LIB
    return build()


if __name__ == "__main__":
    print(build(verbose=True))
