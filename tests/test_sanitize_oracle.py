"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/sanitize/oracle_driver.c calls every oracle entry point on small
inputs with the edge cases the parity tests use (padded strides, masked
rows, repeated and out-of-range ids, NaN and infinite logits, extreme
uniforms, the diagnostics fed by the MC call's outputs).  Built with both
sanitizers and leak detection, any invalid access, leak or undefined
arithmetic aborts the run."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path_factory.mktemp("sanitize") / "oracle_driver")
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-fopenmp", "-Wall", "-Wextra",
           "-o", exe, os.path.join(HERE, "sanitize", "oracle_driver.c"),
           os.path.join(ROOT, "oracle", "opd_oracle.c"), "-lm"]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    return exe


def test_oracle_runs_clean_under_address_and_undefined_behaviour_sanitizers(driver):
    run = subprocess.run([driver], capture_output=True, text=True, env=ENV, timeout=600)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-4000:]
    assert "failures 0" in run.stdout
    assert "ERROR: AddressSanitizer" not in run.stderr
    assert "runtime error" not in run.stderr


def test_the_sanitizer_build_catches_a_planted_overflow(driver):
    run = subprocess.run([driver, "plant-overflow"], capture_output=True, text=True, env=ENV,
                         timeout=120)
    assert run.returncode != 0
    # UndefinedBehaviorSanitizer's object-size check or AddressSanitizer,
    # whichever reaches the read first
    assert "heap-buffer-overflow" in run.stderr or "insufficient space" in run.stderr
