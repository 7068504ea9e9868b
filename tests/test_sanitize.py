"""Host code under AddressSanitizer, UndefinedBehaviorSanitizer and
ThreadSanitizer (CPU only).

* The C oracle, driven over edge inputs by tests/oracle_sanitize_driver.c
  with every input in an allocation of exactly the bytes it may read, so a
  read past a ragged chunk end, an unaligned or overflowing computation, or
  a write past a list cap aborts the run.
* The out-of-band hang-localization library through its own benchmark
  (publications, snapshots idle and under a concurrent writer, torn-read
  count, classification), under ASan/UBSan and, for the lock-free
  publication protocol, under TSan.

Each binary is built with gcc/g++ into a temporary directory; a toolchain
without the sanitizer runtimes skips the test.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "c3_oracle.c")
DRIVER = os.path.join(ROOT, "tests", "oracle_sanitize_driver.c")
OOB_DIR = os.path.join(ROOT, "paper_2608_11034_amd", "csrc", "oob")


def _build(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("sanitizer build unavailable: " + r.stderr.strip()[-300:])


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
    assert "WARNING: ThreadSanitizer" not in r.stderr
    return r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    _build(["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
            "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
            ORACLE_SRC, DRIVER, "-o", exe, "-lm"])
    assert _run(exe).strip().endswith("ok")


def _oob_bench(tmp_path, name, sanitize):
    exe = str(tmp_path / name)
    _build(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", *sanitize,
            os.path.join(OOB_DIR, "c3_oob_bench.cpp"), os.path.join(OOB_DIR, "c3_oob.cpp"),
            "-o", exe, "-lrt", "-pthread"])
    out = _run(exe, "20000")
    assert '"torn": 0' in out, out
    return out


def test_oob_under_asan_ubsan(tmp_path):
    _oob_bench(tmp_path, "oob_asan", ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"])


def test_oob_under_tsan(tmp_path):
    _oob_bench(tmp_path, "oob_tsan", ["-fsanitize=thread"])
