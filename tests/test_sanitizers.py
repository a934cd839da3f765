"""Sanitizer builds of the CPU-side code, run on the CPU.

- The C ABI's host validation (csrc/api.hip) with AddressSanitizer and
  UndefinedBehaviorSanitizer: tests/sanitize/abi_rejections.cpp drives every entry point
  through its rejections (and past validation into stubbed launches), and the build aborts
  on the first undefined behaviour.
- The oracle (oracle/oracle.c) built the same way, under the oracle pin and property tests,
  in a child process that preloads the ASan runtime.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
REPORTS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer", "UndefinedBehaviorSanitizer")


def _clean(out: str):
    for r in REPORTS:
        assert r not in out, out[-4000:]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_validation_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "abi_rejections")
    # host code only is instrumented (each -fsanitize= behind -Xarch_host)
    cmd = [HIPCC, "--offload-arch=gfx950", "-x", "hip", "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2606_24957_amd", "csrc"),
           os.path.join(ROOT, "paper_2606_24957_amd", "csrc", "api.hip"),
           os.path.join(ROOT, "tests", "sanitize", "abi_rejections.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-4000:]
    assert "ok: 0 failed expectations" in out
    _clean(out)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from oracle import build as oracle_build
    lib = oracle_build.build(out=str(tmp_path / "liboracle_asan.so"), sanitize=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    assert os.path.exists(asan), asan
    pre = os.environ.get("LD_PRELOAD", "")
    env = dict(os.environ, DUSTIN_ORACLE_LIB=lib, LD_PRELOAD=asan + (":" + pre if pre else ""),
               ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="4")
    run = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                          os.path.join(ROOT, "tests", "test_oracle_properties.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-4000:]
    assert " passed" in out
    _clean(out)
