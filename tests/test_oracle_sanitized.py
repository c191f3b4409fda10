"""The oracle's CPU pins run again against a build of the same source with
AddressSanitizer and UndefinedBehaviorSanitizer (float-to-integer overflow
included; any finding aborts): out-of-bounds accesses, undefined shifts or
conversions of NaN and infinite values to integers fail this test."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PINS = ["test_oracle_pins.py", "test_oracle_sparse_pins.py", "test_oracle_scale_pins.py", "test_harness_host.py"]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_pins_pass_under_sanitizers(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not installed")
    sys.path.insert(0, ROOT)
    from oracle.build import build
    build(sanitize=True)
    env = dict(os.environ)
    env["EAO_SANITIZE"] = "1"
    env["LD_PRELOAD"] = " ".join([asan, ubsan] + ([env["LD_PRELOAD"]] if env.get("LD_PRELOAD") else []))
    # findings go to log files: pytest holds the test's stderr, which a
    # process the sanitizer stops never gets to print
    log = str(tmp_path / "san")
    env["ASAN_OPTIONS"] = f"detect_leaks=0:abort_on_error=1:verify_asan_link_order=0:log_path={log}"
    env["UBSAN_OPTIONS"] = f"print_stacktrace=1:halt_on_error=1:log_path={log}"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        *[os.path.join(HERE, p) for p in PINS]], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    out = r.stdout + r.stderr
    for f in sorted(tmp_path.glob("san*")):
        out += f"\n--- {f.name}\n" + f.read_text()
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out
