"""The oracle's own pins, rerun on a copy of the oracle built with
AddressSanitizer and UndefinedBehaviorSanitizer (gcc, host code only).

Every out-of-bounds access, use after free, signed overflow, misaligned or
null-pointer use the oracle's tests reach stops the run with a report, so a
green run means the pin suite exercised the oracle without undefined
behaviour.  Leak checking is off: the Python interpreter itself keeps
allocations until exit."""
import glob
import os
import subprocess
import sys

import pytest

from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _runtime(name):
    path = subprocess.check_output(["gcc", f"-print-file-name={name}"], text=True).strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_clean_under_sanitizers(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not installed")
    lib = O.build(out=str(tmp_path / "libtg_oracle_san.so"), extra=SAN)
    tests = sorted(f for f in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py"))
                   if not f.endswith("test_oracle_sanitized.py"))
    env = dict(os.environ)
    env["TG_ORACLE_LIB"] = lib
    # the sanitizer runtimes first (ASan must lead the list), anything already preloaded kept after them
    env["LD_PRELOAD"] = " ".join([asan, ubsan] + ([env["LD_PRELOAD"]] if env.get("LD_PRELOAD") else []))
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    # --capture=sys: a sanitizer report (written to file descriptor 2) reaches the output
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                        "--capture=sys"] + tests,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out
