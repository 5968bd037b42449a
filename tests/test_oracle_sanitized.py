"""The oracle's own pins, re-run against a build of the same C source with
AddressSanitizer and UndefinedBehaviorSanitizer (host code only).  Any
out-of-bounds access, use after free or undefined operation in the oracle
ends the child process with a sanitizer report, and this test fails with
that report."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_oracle_pins_under_address_and_ub_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("libasan not available")
    import oracle
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    tests = sorted(p for p in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py"))
                   if not p.endswith("test_oracle_sanitized.py"))
    env = dict(os.environ, LD_PRELOAD=asan, ORACLE_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:exitcode=86:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    # -s: a sanitizer report goes to the child's stderr, which is kept here
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider", *tests],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    report = "\n".join(ln for ln in (res.stdout + res.stderr).splitlines()
                       if "Sanitizer" in ln or "runtime error" in ln or " in orc_" in ln or "passed" in ln
                       or "failed" in ln)
    assert res.returncode == 0, f"sanitized oracle run failed (exit {res.returncode}):\n{report[-4000:]}"
    assert "Sanitizer" not in res.stderr and "runtime error" not in res.stderr, report[-4000:]
