"""Plain-C host twin of the generator (synth/csrc/gen_host.c), for full-size
workloads where the NumPy twin is too slow.  Bit-identical to
synth.values.unit_values."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import values as V

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libsynth_host.so")
SRC = os.path.join(HERE, "csrc", "gen_host.c")
GCC_FLAGS = ["-O3", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]

_lib = None


def build() -> str:
    subprocess.run(["gcc", *GCC_FLAGS, "-o", LIB + ".tmp", SRC], check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        lib = ctypes.CDLL(LIB)
        lib.synth_host_values.restype = None
        lib.synth_host_values.argtypes = [ctypes.c_uint64, ctypes.c_float, ctypes.c_int,
                                          ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                          ctypes.c_void_p]
        _lib = lib
    return _lib


def unit_values(seed, t, b, scale, dtype, start, count, out=None) -> np.ndarray:
    lib = _load()
    tab = V.normal_table()
    if out is None:
        out = np.empty(count, dtype=np.float32 if dtype == V.DTYPE_F32 else np.uint16)
    lib.synth_host_values(V.unit_key(seed, t, b), float(np.float32(scale)), int(dtype),
                          int(start), int(count), tab.ctypes.data, out.ctypes.data)
    return out
