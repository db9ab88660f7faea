"""ctypes binding of libgnmr (include/gnmr.h): argument marshalling only.

Every computation of the controller pass runs in the HIP library.  Device
pointers are plain ints (``tensor.data_ptr()``); streams are hipStream_t
handles as ints (``torch.cuda.current_stream().cuda_stream``; 0 = null
stream).  If libgnmr.so is missing, loading fails with an error: there is no
fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

# GNMR_LIBRARY names another build of the same library (e.g. a host-sanitizer one)
_LIB_PATH = os.environ.get("GNMR_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libgnmr.so")

GNMR_OK, GNMR_E_INVALID, GNMR_E_NOMEM, GNMR_E_HIP, GNMR_E_STATE = 0, -1, -2, -3, -4
GNMR_F32, GNMR_BF16 = 0, 1
GNMR_BUDGET_ACTIVE, GNMR_BUDGET_ADMITTED, GNMR_BUDGET_STATIC = 0, 1, 2
STATUS_NAMES = {0: "GNMR_OK", -1: "GNMR_E_INVALID", -2: "GNMR_E_NOMEM", -3: "GNMR_E_HIP",
                -4: "GNMR_E_STATE"}

GNMR_FMT_BF16, GNMR_FMT_E2M1, GNMR_FMT_E3M2, GNMR_FMT_E4M3, GNMR_FMT_E5M2, GNMR_FMT_INT8 = \
    0, 1, 2, 3, 4, 5

EXPORTED = ("gnmr_init", "gnmr_destroy", "gnmr_step", "gnmr_step_from_norms", "gnmr_sumsq",
            "gnmr_query", "gnmr_device_outputs", "gnmr_state_size", "gnmr_get_state",
            "gnmr_set_state", "gnmr_set_profiling", "gnmr_profile_read", "gnmr_info",
            "gnmr_last_error", "gnmr_actuator_create", "gnmr_actuate", "gnmr_actuator_info",
            "gnmr_actuator_destroy", "gnmr_wgrad_num_tiles", "gnmr_wgrad_sumsq",
            "gnmr_bind_partials", "gnmr_step_from_partials", "gnmr_wgrad_sumsq_batched",
            "gnmr_actuate_matrix", "gnmr_sumsq_noalloc")
GNMR_NOALLOC_SCRATCH_BYTES = 32 << 20


class GnmrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class gnmr_config(ctypes.Structure):
    _fields_ = [("num_units", ctypes.c_int32), ("window", ctypes.c_int32),
                ("max_o", ctypes.c_int32), ("lock_len", ctypes.c_int32),
                ("eps", ctypes.c_double), ("recoverable", ctypes.c_void_p),
                ("budget_mode", ctypes.c_int32), ("warmup_steps", ctypes.c_int32)]


class gnmr_segments(ctypes.Structure):
    _fields_ = [("num_segments", ctypes.c_int64), ("unit_seg_off", ctypes.c_void_p),
                ("seg_numel", ctypes.c_void_p), ("seg_dtype", ctypes.c_void_p),
                ("seg_ptr", ctypes.c_void_p)]


class gnmr_act_segment(ctypes.Structure):
    _fields_ = [("in_", ctypes.c_void_p), ("out", ctypes.c_void_p), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int32), ("unit", ctypes.c_int32)]


class gnmr_wgrad_problem(ctypes.Structure):
    _fields_ = [("dy", ctypes.c_void_p), ("x", ctypes.c_void_p), ("dw", ctypes.c_void_p),
                ("tokens", ctypes.c_int64), ("out_features", ctypes.c_int32),
                ("in_features", ctypes.c_int32), ("accumulate", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class gnmr_stats(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int64), ("n_trig_gnmr", ctypes.c_int32),
                ("n_trig_dgnmr", ctypes.c_int32), ("n_trig", ctypes.c_int32),
                ("n_cand", ctypes.c_int32), ("n_active", ctypes.c_int32),
                ("hit_maxo", ctypes.c_int32), ("n_nonfinite", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {k: int(getattr(self, k)) for k, _ in self._fields_ if k != "reserved"}


_lib = None


def load_library(path: str = _LIB_PATH) -> ctypes.CDLL:
    """Load libgnmr.so (once).  Raises if it is not built."""
    global _lib
    if _lib is not None and path == _LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    P, I32, I64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    sig = {
        "gnmr_init": [P, P, P, P],
        "gnmr_destroy": [P],
        "gnmr_step": [P, D, D, P, P],
        "gnmr_step_from_norms": [P, P, D, D, P],
        "gnmr_sumsq": [P, P, P, P],
        "gnmr_query": [P, P, P, P, P, P, P, P, P],
        "gnmr_device_outputs": [P, P, P, P, P, P, P, P],
        "gnmr_state_size": [P, P],
        "gnmr_get_state": [P, P, ctypes.c_size_t, P],
        "gnmr_set_state": [P, P, ctypes.c_size_t, P],
        "gnmr_set_profiling": [P, ctypes.c_int],
        "gnmr_profile_read": [P, P, P, P, P],
        "gnmr_info": [P, P, P, P, P],
        "gnmr_actuator_create": [P, P, I64, I32, P],
        "gnmr_actuate": [P, P, I32, I32, P],
        "gnmr_actuate_matrix": [P, P, I64, I32, P, I32, I32, I32, P],
        "gnmr_actuator_info": [P, P, P],
        "gnmr_actuator_destroy": [P],
        "gnmr_wgrad_sumsq": [P, P, P, I64, I32, I32, P, P],
        "gnmr_bind_partials": [P, I64, P],
        "gnmr_wgrad_sumsq_batched": [P, I32, P, P],
        "gnmr_step_from_partials": [P, P, D, D, P],
        "gnmr_sumsq_noalloc": [I32, P, P, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.gnmr_wgrad_num_tiles.argtypes = [I32, I32]
    lib.gnmr_wgrad_num_tiles.restype = I64
    lib.gnmr_last_error.argtypes = []
    lib.gnmr_last_error.restype = ctypes.c_char_p
    if path == _LIB_PATH:
        _lib = lib
    return lib


def _check(status: int) -> None:
    if status != GNMR_OK:
        raise GnmrError(status, load_library().gnmr_last_error().decode())


def _ptr_array(ptrs):
    """Host array of device pointers (ints or objects with data_ptr())."""
    vals = [p.data_ptr() if hasattr(p, "data_ptr") else int(p) for p in ptrs]
    return (ctypes.c_void_p * max(len(vals), 1))(*vals)


def _stream(stream) -> int:
    if stream is None:
        return 0
    return int(getattr(stream, "cuda_stream", stream))


# -- one Python function per C entry point ------------------------------------

def gnmr_init(num_units, window, max_o, lock_len, eps, unit_seg_off, seg_numel, seg_dtype,
              seg_ptr=None, recoverable=None, stream=None, budget_mode=GNMR_BUDGET_ACTIVE,
              warmup_steps=0) -> ctypes.c_void_p:
    lib = load_library()
    uso = np.ascontiguousarray(unit_seg_off, dtype=np.int64)
    numel = np.ascontiguousarray(seg_numel, dtype=np.int64)
    dt = np.ascontiguousarray(seg_dtype, dtype=np.int32)
    rec = None if recoverable is None else np.ascontiguousarray(recoverable, dtype=np.uint8)
    cfg = gnmr_config(int(num_units), int(window), int(max_o), int(lock_len), float(eps),
                      None if rec is None else rec.ctypes.data, int(budget_mode),
                      int(warmup_steps))
    ptrs = None if seg_ptr is None else _ptr_array(seg_ptr)
    segs = gnmr_segments(int(numel.size), uso.ctypes.data, numel.ctypes.data, dt.ctypes.data,
                         None if ptrs is None else ctypes.cast(ptrs, ctypes.c_void_p))
    ctx = ctypes.c_void_p()
    _check(lib.gnmr_init(ctypes.byref(ctx), ctypes.byref(cfg), ctypes.byref(segs),
                         _stream(stream)))
    return ctx


def gnmr_destroy(ctx) -> None:
    _check(load_library().gnmr_destroy(ctx))


def gnmr_step(ctx, alpha_t, beta_t, seg_ptr=None, stream=None) -> None:
    ptrs = None if seg_ptr is None else _ptr_array(seg_ptr)
    _check(load_library().gnmr_step(ctx, float(alpha_t), float(beta_t),
                                    None if ptrs is None else ctypes.cast(ptrs, ctypes.c_void_p),
                                    _stream(stream)))


def gnmr_step_from_norms(ctx, d_norm, alpha_t, beta_t, stream=None) -> None:
    p = d_norm.data_ptr() if hasattr(d_norm, "data_ptr") else int(d_norm)
    _check(load_library().gnmr_step_from_norms(ctx, p, float(alpha_t), float(beta_t),
                                               _stream(stream)))


def gnmr_sumsq(ctx, d_sumsq, seg_ptr=None, stream=None) -> None:
    ptrs = None if seg_ptr is None else _ptr_array(seg_ptr)
    p = d_sumsq.data_ptr() if hasattr(d_sumsq, "data_ptr") else int(d_sumsq)
    _check(load_library().gnmr_sumsq(ctx, None if ptrs is None else ctypes.cast(ptrs, ctypes.c_void_p),
                                     p, _stream(stream)))


def gnmr_sumsq_noalloc(num_units, unit_seg_off, seg_numel, seg_dtype, seg_ptr, d_sumsq,
                       stream=None) -> None:
    uso = np.ascontiguousarray(unit_seg_off, dtype=np.int64)
    numel = np.ascontiguousarray(seg_numel, dtype=np.int64)
    dt = np.ascontiguousarray(seg_dtype, dtype=np.int32)
    ptrs = None if seg_ptr is None else _ptr_array(seg_ptr)
    segs = gnmr_segments(int(numel.size), uso.ctypes.data, numel.ctypes.data, dt.ctypes.data,
                         None if ptrs is None else ctypes.cast(ptrs, ctypes.c_void_p))
    p = d_sumsq.data_ptr() if hasattr(d_sumsq, "data_ptr") else int(d_sumsq)
    _check(load_library().gnmr_sumsq_noalloc(int(num_units), ctypes.byref(segs), p,
                                             _stream(stream)))


def _dptr(p) -> int:
    return p.data_ptr() if hasattr(p, "data_ptr") else int(p)


def gnmr_wgrad_num_tiles(out_features, in_features) -> int:
    return int(load_library().gnmr_wgrad_num_tiles(int(out_features), int(in_features)))


def gnmr_wgrad_sumsq(dy, x, dw, tokens, out_features, in_features, tile_sumsq,
                     stream=None) -> None:
    _check(load_library().gnmr_wgrad_sumsq(_dptr(dy), _dptr(x), _dptr(dw), int(tokens),
                                           int(out_features), int(in_features),
                                           _dptr(tile_sumsq), _stream(stream)))


def gnmr_wgrad_sumsq_batched(problems, tile_sumsq, stream=None) -> None:
    """problems: iterable of (dy, x, dw, tokens, out_features, in_features)
    or (dy, x, dw, tokens, out_features, in_features, accumulate)."""
    ps = []
    for p in problems:
        a, b, c, t, o, i = p[:6]
        acc = int(p[6]) if len(p) > 6 else 0
        ps.append(gnmr_wgrad_problem(_dptr(a), _dptr(b), _dptr(c), int(t), int(o), int(i), acc,
                                     0))
    arr = (gnmr_wgrad_problem * max(len(ps), 1))(*ps)
    _check(load_library().gnmr_wgrad_sumsq_batched(arr, len(ps), _dptr(tile_sumsq),
                                                   _stream(stream)))


def gnmr_bind_partials(ctx, unit_part_off) -> None:
    off = np.ascontiguousarray(unit_part_off, dtype=np.int64)
    _check(load_library().gnmr_bind_partials(ctx, int(off[-1]), off.ctypes.data))


def gnmr_step_from_partials(ctx, d_partial, alpha_t, beta_t, stream=None) -> None:
    _check(load_library().gnmr_step_from_partials(ctx, _dptr(d_partial), float(alpha_t),
                                                  float(beta_t), _stream(stream)))


def gnmr_query(ctx, num_units, stream=None) -> dict:
    U = int(num_units)
    out = {"mask": np.zeros(U, np.uint8), "lock": np.zeros(U, np.int32),
           "norm": np.zeros(U, np.float64), "gnmr": np.zeros(U, np.float64),
           "dgnmr": np.zeros(U, np.float64), "risk": np.zeros(U, np.float64)}
    st = gnmr_stats()
    _check(load_library().gnmr_query(ctx, out["mask"].ctypes.data, out["lock"].ctypes.data,
                                     out["norm"].ctypes.data, out["gnmr"].ctypes.data,
                                     out["dgnmr"].ctypes.data, out["risk"].ctypes.data,
                                     ctypes.byref(st), _stream(stream)))
    out["stats"] = st.as_dict()
    return out


def gnmr_device_outputs(ctx) -> dict:
    ps = [ctypes.c_void_p() for _ in range(7)]
    _check(load_library().gnmr_device_outputs(ctx, *[ctypes.byref(p) for p in ps]))
    names = ("mask", "lock", "norm", "gnmr", "dgnmr", "risk", "stats")
    return {n: p.value for n, p in zip(names, ps)}


def gnmr_state_size(ctx) -> int:
    n = ctypes.c_size_t()
    _check(load_library().gnmr_state_size(ctx, ctypes.byref(n)))
    return n.value


def gnmr_get_state(ctx, stream=None) -> bytes:
    n = gnmr_state_size(ctx)
    buf = ctypes.create_string_buffer(n)
    _check(load_library().gnmr_get_state(ctx, buf, n, _stream(stream)))
    return buf.raw


def gnmr_set_state(ctx, blob: bytes, stream=None) -> None:
    buf = ctypes.create_string_buffer(bytes(blob), len(blob))
    _check(load_library().gnmr_set_state(ctx, buf, len(blob), _stream(stream)))


def gnmr_set_profiling(ctx, enable: bool) -> None:
    _check(load_library().gnmr_set_profiling(ctx, 1 if enable else 0))


def gnmr_profile_read(ctx) -> dict:
    a, b, c = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    n = ctypes.c_int64()
    _check(load_library().gnmr_profile_read(ctx, ctypes.byref(a), ctypes.byref(b),
                                            ctypes.byref(c), ctypes.byref(n)))
    return {"ms_sumsq": a.value, "ms_update": b.value, "ms_select": c.value, "steps": n.value}


def gnmr_info(ctx) -> dict:
    a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    d = ctypes.c_int32()
    _check(load_library().gnmr_info(ctx, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                                    ctypes.byref(d)))
    return {"num_items": a.value, "item_bytes": b.value, "bytes_per_step": c.value,
            "launches_per_step": d.value}


def gnmr_last_error() -> str:
    return load_library().gnmr_last_error().decode()


def gnmr_actuator_create(segments, num_units, stream=None) -> ctypes.c_void_p:
    """segments: iterable of (in, out, rows, cols, unit); in/out are device
    pointers (ints or tensors)."""
    ptr = lambda p: p.data_ptr() if hasattr(p, "data_ptr") else int(p)
    segs = [gnmr_act_segment(ptr(i), ptr(o), int(r), int(c), int(u))
            for i, o, r, c, u in segments]
    arr = (gnmr_act_segment * max(len(segs), 1))(*segs)
    act = ctypes.c_void_p()
    _check(load_library().gnmr_actuator_create(ctypes.byref(act), arr, len(segs), int(num_units),
                                               _stream(stream)))
    return act


def gnmr_actuate(act, d_mask, fmt_low, fmt_recovery, stream=None) -> None:
    p = d_mask.data_ptr() if hasattr(d_mask, "data_ptr") else int(d_mask)
    _check(load_library().gnmr_actuate(act, p, int(fmt_low), int(fmt_recovery), _stream(stream)))


def gnmr_actuate_matrix(x, out, rows, cols, d_mask, unit, fmt_low, fmt_recovery,
                        stream=None) -> None:
    _check(load_library().gnmr_actuate_matrix(_dptr(x), _dptr(out), int(rows), int(cols),
                                              _dptr(d_mask), int(unit), int(fmt_low),
                                              int(fmt_recovery), _stream(stream)))


def gnmr_actuator_info(act) -> dict:
    r, b = ctypes.c_int64(), ctypes.c_int64()
    _check(load_library().gnmr_actuator_info(act, ctypes.byref(r), ctypes.byref(b)))
    return {"rows": r.value, "bytes": b.value}


def gnmr_actuator_destroy(act) -> None:
    _check(load_library().gnmr_actuator_destroy(act))


class Actuator:
    """Recovery actuator over a fixed set of saved-activation segments."""

    def __init__(self, segments, num_units, stream=None):
        self.act = gnmr_actuator_create(segments, num_units, stream)

    def apply(self, d_mask, fmt_low, fmt_recovery, stream=None):
        gnmr_actuate(self.act, d_mask, fmt_low, fmt_recovery, stream)

    def info(self) -> dict:
        return gnmr_actuator_info(self.act)

    def close(self):
        if self.act is not None:
            gnmr_actuator_destroy(self.act)
            self.act = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Controller:
    """One GNMR controller context over a fixed segment layout."""

    def __init__(self, num_units, window, max_o, lock_len, eps, unit_seg_off, seg_numel,
                 seg_dtype, seg_ptr=None, recoverable=None, stream=None,
                 budget_mode=GNMR_BUDGET_ACTIVE, warmup_steps=0):
        self.num_units = int(num_units)
        self.ctx = gnmr_init(num_units, window, max_o, lock_len, eps, unit_seg_off, seg_numel,
                             seg_dtype, seg_ptr, recoverable, stream, budget_mode, warmup_steps)

    def step(self, alpha_t, beta_t, seg_ptr=None, stream=None):
        gnmr_step(self.ctx, alpha_t, beta_t, seg_ptr, stream)

    def step_from_norms(self, d_norm, alpha_t, beta_t, stream=None):
        gnmr_step_from_norms(self.ctx, d_norm, alpha_t, beta_t, stream)

    def sumsq(self, d_sumsq, seg_ptr=None, stream=None):
        gnmr_sumsq(self.ctx, d_sumsq, seg_ptr, stream)

    def bind_partials(self, unit_part_off):
        if len(unit_part_off) != self.num_units + 1:
            raise ValueError(f"unit_part_off needs num_units + 1 = {self.num_units + 1} entries")
        gnmr_bind_partials(self.ctx, unit_part_off)

    def step_from_partials(self, d_partial, alpha_t, beta_t, stream=None):
        gnmr_step_from_partials(self.ctx, d_partial, alpha_t, beta_t, stream)

    def query(self, stream=None) -> dict:
        return gnmr_query(self.ctx, self.num_units, stream)

    def device_outputs(self) -> dict:
        return gnmr_device_outputs(self.ctx)

    def get_state(self, stream=None) -> bytes:
        return gnmr_get_state(self.ctx, stream)

    def set_state(self, blob, stream=None):
        gnmr_set_state(self.ctx, blob, stream)

    def set_profiling(self, enable=True):
        gnmr_set_profiling(self.ctx, enable)

    def profile_read(self) -> dict:
        return gnmr_profile_read(self.ctx)

    def info(self) -> dict:
        return gnmr_info(self.ctx)

    def close(self):
        if self.ctx is not None:
            gnmr_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
