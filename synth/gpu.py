"""Driver of the HIP generator (libsynth_gen.so): fills a device buffer laid
out by synth.layout with the values defined in synth.values."""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import values as V

_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth_gen.so")


class _Job(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("numel", ctypes.c_int64),
                ("unit_base", ctypes.c_int64), ("key", ctypes.c_uint64),
                ("scale", ctypes.c_float), ("dtype", ctypes.c_int32)]


class Generator:
    """Holds the normal table on the device and the loaded library."""

    def __init__(self, device="cuda"):
        import torch

        if not os.path.exists(_LIB):
            raise RuntimeError(f"{_LIB} is not built (run __graft_entry__.build())")
        self.lib = ctypes.CDLL(_LIB)
        self.lib.synth_fill.restype = ctypes.c_int
        self.lib.synth_fill.argtypes = [ctypes.POINTER(_Job), ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_void_p]
        self.table = torch.from_numpy(V.normal_table().copy()).to(device)

    def fill(self, layout, base_ptr: int, seed: int, t: int, scale32, units=None,
             stream: int = 0) -> None:
        """Write step t's values of the given units (default all) into the
        buffer at base_ptr; scale32[b] is unit b's fp32 scale."""
        scale32 = np.asarray(scale32, dtype=np.float32)
        sel = range(layout.num_units) if units is None else units
        jobs = []
        for b in sel:
            key = V.unit_key(seed, t, int(b))
            for s in range(layout.unit_seg_off[b], layout.unit_seg_off[b + 1]):
                if layout.seg_numel[s] == 0:
                    continue
                jobs.append(_Job(base_ptr + int(layout.seg_byte_off[s]), int(layout.seg_numel[s]),
                                 int(layout.seg_unit_base[s]), key, float(scale32[b]),
                                 int(layout.seg_dtype[s])))
        if not jobs:
            return
        arr = (_Job * len(jobs))(*jobs)
        rc = self.lib.synth_fill(arr, len(jobs), self.table.data_ptr(), stream)
        if rc != 0:
            raise RuntimeError(f"synth_fill failed with hipError {rc}")


class ReadProbe:
    """Plain read-reduce kernels over a contiguous device buffer (the
    benchmark's read-ceiling reference points): variant 0 is a grid-stride
    loop, variant 1 one 64 KiB block per workgroup in XCD-contiguous order;
    and a plain copy, the read-and-write reference."""

    VARIANTS = {0: "grid_stride_nt", 1: "blocked_nt_xcd"}

    def __init__(self):
        if not os.path.exists(_LIB):
            raise RuntimeError(f"{_LIB} is not built (run __graft_entry__.build())")
        self.lib = ctypes.CDLL(_LIB)
        self.lib.synth_read_probe_partials.restype = ctypes.c_int64
        self.lib.synth_read_probe_partials.argtypes = [ctypes.c_int64, ctypes.c_int32]
        self.lib.synth_read_probe.restype = ctypes.c_int
        self.lib.synth_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                              ctypes.c_int32, ctypes.c_void_p]
        self.lib.synth_copy_probe.restype = ctypes.c_int
        self.lib.synth_copy_probe.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                              ctypes.c_void_p]

    def num_partials(self, nbytes: int, variant: int) -> int:
        return int(self.lib.synth_read_probe_partials(int(nbytes), int(variant)))

    def run(self, ptr: int, nbytes: int, partials_ptr: int, variant: int, stream: int = 0):
        rc = self.lib.synth_read_probe(ptr, int(nbytes), partials_ptr, int(variant), stream)
        if rc != 0:
            raise RuntimeError(f"synth_read_probe failed with hipError {rc}")

    def copy(self, src_ptr: int, dst_ptr: int, nbytes: int, stream: int = 0):
        """The read-and-write reference: a plain non-temporal copy."""
        rc = self.lib.synth_copy_probe(src_ptr, dst_ptr, int(nbytes), stream)
        if rc != 0:
            raise RuntimeError(f"synth_copy_probe failed with hipError {rc}")
