"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The oracle's C source is built again with the oracle's own gcc flags plus
-fsanitize=address,undefined, and the oracle pin tests run against that build
in a subprocess whose Python loads the sanitizer runtimes first.  Any
out-of-bounds access, use after free or undefined operation (signed overflow,
an over-wide shift) in the oracle aborts the run, so the test fails.  The
host-side validation of the oracle's entry points (sizes, NULL pointers) is
exercised by the same pin tests.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

PIN_TESTS = ["tests/test_oracle_worked.py", "tests/test_oracle_quantize_pack.py",
             "tests/test_oracle_conv_dense.py", "tests/test_oracle_encodings.py"]


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=" + name],
                          capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_pass_under_sanitizers(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("gcc sanitizer runtimes not installed")
    for f in ("bsref.c", "bsref.h"):
        shutil.copy(os.path.join(ROOT, "oracle", f), tmp_path / f)
    lib = str(tmp_path / "libbsref_san.so")
    subprocess.run(
        ["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared",
         "-ffp-contract=off", "-fno-fast-math", "-fno-omit-frame-pointer",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
         str(tmp_path / "bsref.c"), "-o", lib, "-lm"],
        check=True, cwd=str(tmp_path))
    env = dict(os.environ, BSREF_LIBRARY=lib, LD_PRELOAD=asan + ":" + ubsan,
               # Python's own allocations are not the oracle's to report
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
         "-m", "not gpu and not slow"] + PIN_TESTS,
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    assert "ERROR: AddressSanitizer" not in out, out[-3000:]
    assert "runtime error:" not in out, out[-3000:]
