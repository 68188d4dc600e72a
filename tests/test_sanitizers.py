"""Sanitizer runs on the CPU (no GPU needed):

* the oracle (oracle.c) built with gcc under AddressSanitizer and
  UndefinedBehaviorSanitizer, driven over edge-case shapes by
  tests/sanitize/oracle_check.c on buffers of exactly the documented sizes;
* the library's host code (argument validation, kernel selection, launch
  set-up) built with host-side AddressSanitizer and UndefinedBehaviorSanitizer
  (device code as usual), loaded into a child process with the sanitizer
  runtime preloaded, running the boundary and plan tests.

Either run aborts on the first error the sanitizers find.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_under_asan_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_check")
    cmd = ["gcc", "-std=c99", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", exe,
           os.path.join(ROOT, "oracle", "oracle.c"),
           os.path.join(ROOT, "tests", "sanitize", "oracle_check.c"), "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", OMP_NUM_THREADS="4")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ran clean" in r.stdout


def _sanitized_library():
    from paper_1802_04647_amd import build
    srcs = glob.glob(os.path.join(ROOT, "paper_1802_04647_amd", "csrc", "*")) + \
        glob.glob(os.path.join(ROOT, "include", "*.h"))
    newest = max(os.path.getmtime(p) for p in srcs)
    if not os.path.exists(build.SAN_LIB) or os.path.getmtime(build.SAN_LIB) < newest:
        build.build(sanitize=True)
    return build.SAN_LIB, build.sanitizer_runtime()


def test_host_code_under_asan_ubsan():
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("runs on CPU hosts: the child process must not initialise a GPU")
    try:
        lib, rt = _sanitized_library()
    except (RuntimeError, OSError) as e:
        pytest.skip(f"sanitized build unavailable: {e}")
    if not rt or not os.path.exists(rt):
        pytest.skip("AddressSanitizer runtime not found")
    env = dict(os.environ, LD_PRELOAD=rt, DMLNN_LIBRARY=lib, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p",
                        "no:cacheprovider", os.path.join(ROOT, "tests", "test_boundary.py"),
                        os.path.join(ROOT, "tests", "test_plan.py")],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out
