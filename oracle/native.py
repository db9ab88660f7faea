"""Plain-C sum of squares of the oracle (oracle/csrc/sumsq.c) -- TEST
INFRASTRUCTURE ONLY.  The same definition as oracle.sumsq: exact widening,
exact squares, float64 additions (here in index order)."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libgnmr_oracle.so")
SRC = os.path.join(HERE, "csrc", "sumsq.c")
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
        for name in ("oracle_sumsq_f32", "oracle_sumsq_bf16"):
            fn = getattr(lib, name)
            fn.restype = ctypes.c_double
            fn.argtypes = [ctypes.c_void_p, ctypes.c_int64]
        _lib = lib
    return _lib


def sumsq(values: np.ndarray, dtype: int) -> float:
    """dtype 0 = fp32 values, 1 = bf16 given as uint16 bit patterns."""
    lib = _load()
    if dtype == 0:
        x = np.ascontiguousarray(values, dtype=np.float32)
        return lib.oracle_sumsq_f32(x.ctypes.data, x.size)
    if dtype == 1:
        x = np.ascontiguousarray(values, dtype=np.uint16)
        return lib.oracle_sumsq_bf16(x.ctypes.data, x.size)
    raise ValueError(f"unknown dtype {dtype}")
