"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The C oracle, linked with `sanitize_oracle.c`: every quantizer on ragged,
  strided, non-finite inputs with exactly sized output buffers, plus the scalar
  codecs at their extremes.
* The C ABI's host side (`csrc/api.hip` compiled for the host only), linked
  with `sanitize_api.cpp`, whose stub launchers stand in for the kernels: valid
  and invalid calls of every entry point, including sizes and strides large
  enough to overflow unchecked 64-bit layout arithmetic.

Each driver exits non-zero on a sanitizer report or a failed check.  The GPU
code is not built here: the device side has no sanitizer on this target.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2607_24953_amd", "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, exe):
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr[-4000:]
    run = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "Sanitizer" not in run.stderr, run.stderr[-4000:]
    return run.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_oracle")
    cmd = ["gcc", "-std=c99", "-g", "-O1", "-fno-omit-frame-pointer", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", exe,
           os.path.join(HERE, "sanitize_oracle.c"), os.path.join(ROOT, "oracle", "q2d_oracle.c"), "-lm"]
    assert "sanitize_oracle: ok" in _run(cmd, exe)


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    return None


@pytest.mark.skipif(_hipcc() is None, reason="hipcc not found")
def test_abi_host_side_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_api")
    # host-only compilation; each sanitizer flag is scoped to the host pass
    cmd = [_hipcc(), "-x", "hip", "--cuda-host-only", "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "api.hip"), os.path.join(HERE, "sanitize_api.cpp"), "-o", exe]
    assert "sanitize_api: ok" in _run(cmd, exe)
