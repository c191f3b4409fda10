"""The host ABI and benchmark host tests run again against the library's host code built with
AddressSanitizer and UndefinedBehaviorSanitizer (any finding aborts): the
argument checks, the quantizer validation fuzz, the message and workspace
size arithmetic and the launch planning reach no out-of-bounds access, no
signed overflow, no undefined shift or conversion."""
import glob
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _clang_asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_abi_host_tests_pass_under_sanitizers(tmp_path):
    rt = _clang_asan_runtime()
    if rt is None:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    sys.path.insert(0, ROOT)
    from paper_2205_14473_amd.build import build_host_sanitized
    try:
        lib = build_host_sanitized(str(tmp_path / "san"))
    except FileNotFoundError as e:
        pytest.skip(str(e))
    log = str(tmp_path / "findings")
    env = dict(os.environ)
    env["EA_LIB"] = lib
    env["LD_PRELOAD"] = " ".join([rt] + ([env["LD_PRELOAD"]] if env.get("LD_PRELOAD") else []))
    env["ASAN_OPTIONS"] = f"detect_leaks=0:abort_on_error=1:verify_asan_link_order=0:log_path={log}"
    env["UBSAN_OPTIONS"] = f"print_stacktrace=1:halt_on_error=1:log_path={log}"
    # the sanitized build is the one the binding loads
    r = subprocess.run([sys.executable, "-c", "import paper_2205_14473_amd._binding as b; print(b.LIB_PATH)"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == lib, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(HERE, "test_abi_host.py"), os.path.join(HERE, "test_bench_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    out = r.stdout + r.stderr
    for f in sorted(tmp_path.glob("findings*")):
        out += f"\n--- {f.name}\n" + f.read_text()
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out
