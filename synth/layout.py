"""Placement of a workload's units as segments of one flat device buffer.

A unit is one or more segments; the generator numbers a unit's elements
across its segments in order, and the controller's unit norm is over the
concatenation.  Offsets are in bytes from the start of the buffer."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .values import DTYPE_SIZE


@dataclass
class Layout:
    unit_seg_off: np.ndarray   # int64 [U+1]
    seg_numel: np.ndarray      # int64 [S]
    seg_dtype: np.ndarray      # int32 [S]
    seg_unit: np.ndarray       # int64 [S]
    seg_unit_base: np.ndarray  # int64 [S], first element of the segment inside its unit
    seg_byte_off: np.ndarray   # int64 [S]
    total_bytes: int

    @property
    def num_units(self) -> int:
        return len(self.unit_seg_off) - 1

    @property
    def num_segments(self) -> int:
        return len(self.seg_numel)

    def unit_numel(self) -> np.ndarray:
        out = np.zeros(self.num_units, dtype=np.int64)
        np.add.at(out, self.seg_unit, self.seg_numel)
        return out


def build(unit_numel, unit_dtype, pieces=None, align: int = 256, shift=None) -> Layout:
    """pieces[b]: list of segment lengths of unit b (default: one segment);
    shift[s]: extra byte offset (a multiple of the element size) added before
    segment s, to place segments at arbitrary alignments."""
    unit_numel = np.asarray(unit_numel, dtype=np.int64)
    unit_dtype = np.asarray(unit_dtype, dtype=np.int32)
    U = unit_numel.size
    off = [0]
    numel, dtype, unit, base, boff = [], [], [], [], []
    pos = 0
    s = 0
    for b in range(U):
        lens = [int(unit_numel[b])] if pieces is None else [int(x) for x in pieces[b]]
        assert sum(lens) == unit_numel[b]
        e = 0
        for n in lens:
            esz = DTYPE_SIZE[int(unit_dtype[b])]
            pos = (pos + align - 1) // align * align
            if shift is not None:
                pos += int(shift[s])
                assert pos % esz == 0
            numel.append(n)
            dtype.append(int(unit_dtype[b]))
            unit.append(b)
            base.append(e)
            boff.append(pos)
            pos += n * esz
            e += n
            s += 1
        off.append(s)
    return Layout(np.array(off, np.int64), np.array(numel, np.int64), np.array(dtype, np.int32),
                  np.array(unit, np.int64), np.array(base, np.int64), np.array(boff, np.int64),
                  (pos + align - 1) // align * align)


def for_workload(w, align: int = 256) -> Layout:
    pieces = None
    if any(u.pieces for u in w.units):
        pieces = [list(u.pieces) if u.pieces else [u.numel] for u in w.units]
    return build(w.numel, w.dtypes, pieces=pieces, align=align)
