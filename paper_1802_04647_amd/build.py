"""Build libdmlnn.so (the HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_1802_04647_amd.build

Objects go to ``_build/`` at the repository root; the shared library is written
next to this file, where the binding loads it.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(ROOT, "_build", "dmlnn")
LIB = os.path.join(HERE, "libdmlnn.so")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
ARCH = "gfx950"
# Packed fp32 VALU ops are disabled for all device code (the compiler would
# otherwise fuse pairs of float operations into them).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
CFLAGS = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", f"--offload-arch={ARCH}", "-Wall",
          "-Wno-unused-command-line-argument", *DEVICE_FLAGS]


# Host-side AddressSanitizer + UndefinedBehaviorSanitizer (the host code only:
# argument validation, plan selection, launch set-up; device code is built as
# usual).  The sanitized copy is for the CPU tests; it needs the sanitizer
# runtime preloaded into the process that loads it.
SAN_DIR = os.path.join(ROOT, "_build", "dmlnn_san")
SAN_LIB = os.path.join(SAN_DIR, "libdmlnn.so")
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _compile(src: str, out_dir: str = OUT_DIR, extra=()) -> str:
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    out_dir, lib = (SAN_DIR, SAN_LIB) if sanitize else (OUT_DIR, LIB)
    extra = SAN_FLAGS if sanitize else []
    os.makedirs(out_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    jobs = min(len(srcs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, out_dir, extra), srcs))
    tmp = lib + ".tmp"
    link_san = ["-shared-libasan", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
                "-fsanitize=undefined"] if sanitize else []
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_san, "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib} from {len(srcs)} sources")
    return lib


def sanitizer_runtime() -> str:
    """Path of the AddressSanitizer runtime the sanitized library links against."""
    clang = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True)
    return r.stdout.strip()


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
