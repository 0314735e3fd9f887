"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/oracle_sanitize_driver.c includes oracle/mx_oracle.c and calls every
entry point on small odd shapes with special values; built here with gcc
-fsanitize=address,undefined and no recovery, any out-of-bounds access,
overflow or invalid shift in the oracle fails the run.  Host code only: the
HIP path is not involved.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _sanitizers_available(tmp):
    probe = os.path.join(tmp, "probe.c")
    with open(probe, "w") as f:
        f.write("int main(void) { return 0; }\n")
    r = subprocess.run(["gcc", "-fsanitize=address,undefined", probe, "-o",
                        os.path.join(tmp, "probe")], capture_output=True)
    return r.returncode == 0


def test_oracle_clean_under_asan_and_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    tmp = str(tmp_path)
    if not _sanitizers_available(tmp):
        pytest.skip("gcc has no sanitizer runtime here")
    exe = os.path.join(tmp, "oracle_sanitize")
    build = subprocess.run(
        ["gcc", "-std=c99", "-O1", "-g", "-ffp-contract=off", "-fno-fast-math",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         os.path.join(HERE, "oracle_sanitize_driver.c"), "-o", exe, "-lm"],
        capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stderr[-4000:]
    assert "runtime error" not in run.stderr, run.stderr[-4000:]
    assert "oracle sanitizer run: ok" in run.stdout
