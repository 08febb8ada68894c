"""The CPU oracle and the input generator under AddressSanitizer and
UndefinedBehaviorSanitizer (no GPU): tests/sanitize_driver.c drives every
entry point of oracle/raas_oracle.c and synth/raas_synth.c through the
configurations the parity tests use; a sanitizer report fails the test."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_and_generator_under_sanitizers(tmp_path):
    exe = str(tmp_path / "sanitize_driver")
    cmd = ["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fopenmp", os.path.join(HERE, "sanitize_driver.c"), oracle.SRC,
           os.path.join(ROOT, "synth", "raas_synth.c"), "-lm", "-o", exe]
    subprocess.check_call(cmd)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    res = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=900)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-6000:]
    assert "ok" in res.stdout
