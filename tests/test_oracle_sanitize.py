"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer and
driven through every entry point on small seeded shapes (tests/sanitize/
oracle_driver.c): no out-of-bounds access, leak, signed overflow or other
undefined behaviour is reported.  Skipped where gcc has no sanitizer runtime."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "oracle", "sq_oracle.c"), os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c")]
FLAGS = ["-O1", "-g", "-std=c99", "-fno-fast-math", "-ffp-contract=off", "-fno-omit-frame-pointer",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    r = subprocess.run(["gcc", *FLAGS, *SRC, "-o", exe, "-lm"], capture_output=True, text=True)
    if r.returncode != 0:
        if "asan" in r.stderr or "ubsan" in r.stderr or "sanitize" in r.stderr:
            pytest.skip("gcc without sanitizer runtimes: " + r.stderr[-300:])
        raise AssertionError(r.stderr)
    # verify_asan_link_order=0: the environment may preload other libraries ahead of the runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0 and run.stdout.strip() == "ok", run.stderr[-2000:]
    assert "runtime error" not in run.stderr and "ERROR: AddressSanitizer" not in run.stderr, run.stderr[-2000:]
