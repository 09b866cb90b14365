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


def _asan_runtime():
    import glob
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(_asan_runtime() is None or not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc or its AddressSanitizer runtime not found")
def test_host_code_under_address_sanitizer(tmp_path):
    """The library's host code (C ABI, argument checks, handle bookkeeping,
    the batch handoff) built with AddressSanitizer -- host side only, the
    gfx950 kernels are built as usual -- and the CPU tests that call it run
    against that build (HS_LIBRARY)."""
    csrc = os.path.join(ROOT, "paper_2603_12707_amd", "csrc")
    objs, procs = [], []
    for f in ("hs_api.cpp", "hs_gemm.hip", "hs_attn.hip", "hs_misc.hip", "hs_handoff.cpp"):
        obj = str(tmp_path / (f + ".o"))
        cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer",
               "-I", os.path.join(ROOT, "include"), "-c", "-x", "hip", os.path.join(csrc, f), "-o", obj]
        procs.append(subprocess.Popen(cmd, stderr=subprocess.DEVNULL))
        objs.append(obj)
    for p in procs:
        assert p.wait() == 0
    lib = str(tmp_path / "libhs_asan.so")
    subprocess.check_call(["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-shared", "-fPIC",
                           "-Xarch_host", "-fsanitize=address", "-shared-libasan", "-o", lib] + objs)
    env = dict(os.environ, HS_LIBRARY=lib, LD_PRELOAD=_asan_runtime(), ASAN_OPTIONS="detect_leaks=0")
    r = subprocess.run(["python", "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_handoff.py"), os.path.join(ROOT, "tests", "test_abi.py")],
                       capture_output=True, text=True, timeout=600, env=env, cwd=ROOT)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "AddressSanitizer" not in r.stderr, r.stderr[-3000:]
