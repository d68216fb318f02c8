"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer (gcc, host
code only) and driven over every function and its edge cases by
tests/oracle_sanitize_driver.c: no memory error or undefined behaviour may occur."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not installed")
    exe = tmp_path / "oracle_sanitized"
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fno-fast-math", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "oracle"),
           os.path.join(ROOT, "tests", "oracle_sanitize_driver.c"), os.path.join(ROOT, "oracle", "monomoe_oracle.c"),
           "-lm", "-o", str(exe)]
    cc = subprocess.run(cmd, capture_output=True, text=True)
    if cc.returncode != 0 and "cannot find" in cc.stderr and "asan" in cc.stderr:
        pytest.skip("sanitizer runtime not installed: " + cc.stderr.strip().splitlines()[-1])
    assert cc.returncode == 0, cc.stderr
    # verify_asan_link_order=0: the environment may preload other libraries before the ASan runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout + run.stderr
    assert run.stdout.strip() == "ok"
