"""Registers a PyTorch model's parameter gradients as GNMR units.

Each unit is the set of parameters that `unit_of(name)` maps to one key
(default: every parameter is its own unit; mapping a whole block's parameters
to one key gives the block-as-unit granularity of Sec. 3.4).  A unit's
segments are its parameters' `.grad` tensors, in registration order.  The
gradient pointers are passed to the library on every step, because
`zero_grad(set_to_none=True)` reallocates `.grad` buffers.

Argument marshalling only: the controller pass runs in libgnmr.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np

from .binding import GNMR_BF16, GNMR_BUDGET_ACTIVE, GNMR_F32, Controller

LLAMA_LINEARS = ("q_proj", "k_proj", "v_proj", "o_proj", "gate_proj", "up_proj", "down_proj")


def llama_linear_units(name: str):
    """Default unit map for LLaMA-style models: each attention / SwiGLU
    projection weight is one recoverable unit (Sec. 2 operator view); other
    parameters are not monitored."""
    parts = name.split(".")
    if len(parts) >= 2 and parts[-1] == "weight" and parts[-2] in LLAMA_LINEARS:
        return ".".join(parts[:-1])
    return None


class TorchUnits:
    def __init__(self, named_parameters, window: int = 5, max_o: int = 8, lock_len: int = 8,
                 eps: float = 1e-12, unit_of=lambda name: name, recoverable=None,
                 budget_mode: int = GNMR_BUDGET_ACTIVE, warmup_steps: int = 0, stream=None):
        import torch

        groups = OrderedDict()
        for name, p in named_parameters:
            key = unit_of(name)
            if key is None or not p.requires_grad:
                continue
            if p.dtype not in (torch.bfloat16, torch.float32):
                raise TypeError(f"{name}: only bf16 and fp32 gradients are supported")
            groups.setdefault(key, []).append((name, p))
        if not groups:
            raise ValueError("no parameter was mapped to a unit")
        self.unit_names = list(groups.keys())
        self.params = [p for ps in groups.values() for _, p in ps]
        self.param_names = [n for ps in groups.values() for n, _ in ps]
        off = np.zeros(len(groups) + 1, dtype=np.int64)
        off[1:] = np.cumsum([len(ps) for ps in groups.values()])
        numel = [p.numel() for p in self.params]
        dtype = [GNMR_BF16 if p.dtype == torch.bfloat16 else GNMR_F32 for p in self.params]
        rec = None
        if recoverable is not None:
            rec = np.array([1 if recoverable(u) else 0 for u in self.unit_names], np.uint8)
        self.ctl = Controller(len(groups), window, max_o, lock_len, eps, off, numel, dtype,
                              None, rec, stream, budget_mode, warmup_steps)

    def grad_pointers(self):
        ptrs = []
        for name, p in zip(self.param_names, self.params):
            g = p.grad
            if g is None:
                raise RuntimeError(f"{name}.grad is None; run backward before the controller step")
            if not g.is_contiguous() or g.dtype != p.dtype or g.device != p.device:
                raise RuntimeError(f"{name}.grad must be a contiguous {p.dtype} tensor on {p.device}")
            ptrs.append(g.data_ptr())
        return ptrs

    def step(self, alpha_t: float, beta_t: float, stream=None) -> None:
        """One controller step over the current gradients (asynchronous)."""
        self.ctl.step(alpha_t, beta_t, seg_ptr=self.grad_pointers(), stream=stream)

    def query(self, stream=None) -> dict:
        out = self.ctl.query(stream)
        out["units"] = self.unit_names
        return out

    def recovery_set(self, stream=None) -> list:
        """Names of the units on the recovery path after the last step (A_t)."""
        m = self.ctl.query(stream)["mask"]
        return [u for u, a in zip(self.unit_names, m) if a]

    def close(self):
        self.ctl.close()
