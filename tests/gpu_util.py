"""Helpers of the GPU tests: device buffers for a layout, step comparison."""
from __future__ import annotations

import numpy as np


def require_gpu():
    import torch

    assert torch.cuda.is_available(), "this test needs an MI355X (HIP device)"
    return torch


def device_buffer(torch, layout):
    buf = torch.empty(max(layout.total_bytes, 256), dtype=torch.uint8, device="cuda")
    base = buf.data_ptr()
    ptrs = [base + int(o) for o in layout.seg_byte_off]
    return buf, base, ptrs


def controller_for(layout, w=None, ptrs=None, **cfg):
    from paper_2606_00539_amd import Controller

    if w is not None:
        cfg = dict(dict(window=w.window, max_o=w.max_o, lock_len=w.lock_len, eps=w.eps), **cfg)
    return Controller(layout.num_units, cfg.pop("window"), cfg.pop("max_o"), cfg.pop("lock_len"),
                      cfg.pop("eps"), layout.unit_seg_off, layout.seg_numel, layout.seg_dtype,
                      ptrs, **cfg)


def assert_step_matches(out, ref, rtol=1e-5, what=""):
    """Masks, locks and counters bit-exact; norms and ratios within rtol."""
    bad = np.flatnonzero(out["mask"] != ref.mask)
    assert bad.size == 0, f"{what} mask differs at units {bad[:10]}"
    bad = np.flatnonzero(out["lock"] != ref.lock)
    assert bad.size == 0, f"{what} lock differs at units {bad[:10]}"
    for k, v in ref.stats.items():
        assert out["stats"][k] == v, f"{what} stats[{k}] {out['stats'][k]} != {v}"
    for f in ("norm", "gnmr", "dgnmr", "risk"):
        np.testing.assert_allclose(out[f], getattr(ref, f), rtol=rtol, atol=0,
                                   err_msg=f"{what} {f}")
