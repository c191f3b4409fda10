"""Compile the C oracle into ``oracle/liboracle.so`` with gcc.

Test infrastructure only: the product library never links this object.
``-ffp-contract=off`` keeps every a*b+c as two binary32 roundings; no
fast-math flag is used, so division and square root are correctly rounded.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
SAN_LIB = os.path.join(HERE, "liboracle_san.so")
SOURCES = [os.path.join(HERE, "eao.c")]
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-fno-strict-aliasing", "-Wall", "-Wextra"]
# The same source checked by AddressSanitizer and UndefinedBehaviorSanitizer
# (with float-to-integer overflow, which -fsanitize=undefined leaves out);
# any finding aborts.  Loaded instead of LIB when EAO_SANITIZE=1, into a
# process that preloads the sanitizer runtimes.
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fsanitize=float-cast-overflow", "-fno-sanitize-recover=all"]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile the oracle; returns the path of the shared object."""
    out = SAN_LIB if sanitize else LIB
    flags = [f for f in CFLAGS if not (sanitize and f == "-O2")] + (SAN_FLAGS if sanitize else [])
    cmd = ["gcc", *flags, *SOURCES, "-lm", "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def ensure_built() -> str:
    """Build only when the shared object is missing or older than a source.

    EAO_LIB, when set, names a library to load instead, built elsewhere from
    a copy of the source (the mutation test plants one mistake in each copy
    and runs the pins against it)."""
    override = os.environ.get("EAO_LIB")
    if override:
        if not os.path.exists(override):
            raise FileNotFoundError(f"EAO_LIB={override} does not exist")
        return override
    sanitize = os.environ.get("EAO_SANITIZE") == "1"
    lib = SAN_LIB if sanitize else LIB
    if os.path.exists(lib):
        t = os.path.getmtime(lib)
        srcs = SOURCES + [os.path.join(HERE, "eao.h")]
        if all(os.path.getmtime(s) <= t for s in srcs):
            return lib
    return build(sanitize=sanitize)


if __name__ == "__main__":
    print(build(verbose=True))
