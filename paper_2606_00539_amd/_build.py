"""Builds libgnmr.so in-tree with hipcc for gfx950."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libgnmr.so")
SOURCES = [os.path.join(PKG, "csrc", f)
           for f in ("gnmr_runtime.hip", "k1_sumsq.hip", "k23_control.hip", "k4_actuator.hip",
                     "k5_wgrad.hip")]
HEADERS = [os.path.join(PKG, "csrc", f) for f in ("gnmr_internal.h", "k1_geometry.h")] + [
    os.path.join(ROOT, "include", "gnmr.h")]

# Packed-fp32 instructions are switched off for all device code.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = True) -> str:
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"),
           "-o", LIB + ".tmp", *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


# AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (the
# device code is built as usual); any undefined behaviour aborts.
HOST_SANITIZE_FLAGS = ["-O1", "-g", "-shared-libsan",
                       "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                       "-Xarch_host", "-fno-sanitize-recover=undefined",
                       "-Xarch_host", "-fno-omit-frame-pointer"]


def sanitizer_runtime():
    """The clang AddressSanitizer runtime that a process loading the
    host-sanitized library must preload, or None if this toolchain has none."""
    import glob

    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    found = sorted(glob.glob(os.path.join(rocm, "llvm", "lib", "clang", "*", "lib", "linux",
                                          "libclang_rt.asan-x86_64.so")))
    return found[-1] if found else None


def build_host_sanitized(out_path: str) -> str:
    """libgnmr.so with the host code under the sanitizers, at out_path (for
    CPU tests of the host logic: argument checks, work lists, overlap checks,
    error paths)."""
    cmd = [hipcc(), *HIPCC_FLAGS, *HOST_SANITIZE_FLAGS, "-I", os.path.join(ROOT, "include"),
           "-o", out_path, *SOURCES]
    subprocess.run(cmd, check=True, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE)
    return out_path


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
