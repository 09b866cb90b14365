"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
and driven through every entry point (tests/asan/oracle_asan.c): small models of
each storage dtype and RoPE kind, with and without q/k/v bias and LM head,
prefill, decode to capacity, a cache copied row by row, and the argument and
state errors.  Any out-of-bounds access, leak or undefined behaviour fails the
run."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    subprocess.check_call(["gcc", "-std=c11", "-g", "-O1", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-Wall", "-Werror",
                           "-I", os.path.join(ROOT, "oracle"), os.path.join(ROOT, "oracle", "hs_oracle.c"),
                           os.path.join(ROOT, "tests", "asan", "oracle_asan.c"), "-lm", "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.strip() == "ok"
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
