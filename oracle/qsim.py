"""Oracle of the quantisation-simulated linear operator -- TEST INFRASTRUCTURE
ONLY (same rules as the rest of oracle/: only tests/, __graft_entry__.smoke()
and bench.py's cpu_baseline leg may use it; it shares nothing with the HIP
library or its binding).

What it computes (App. E.2, quantisation-simulated low-precision operators):
a bias-free linear layer y = x w^T whose tensors are fake-quantised --
scaled into the target format's range, rounded to its nearest representable
value and scaled back -- at each point the paper names:

  forward   x_q = Q(x), w_q = Q(w), y = x_q w_q^T, output y_q = Q(y)
  backward  dy_q = Q(dy), dx = dy_q w_q, dx_q = Q(dx) (passed on),
            dw = dy_q^T x_q, dw_q = Q(dw) (the weight gradient)

The format follows the unit's controller decision (Alg. 2): the low-cost
formats when the unit is outside A_t, the recovery formats when it is in A_t,
each with one format for the forward quantisations and one for the backward
ones (the paper's recovery path is hybrid FP8: E4M3 forward, E5M2 backward).

Readings (the paper gives the per-token recipe for activations only):
  * every quantisation is the per-row recipe of oracle/fakequant.py
    (fakequant_rows): rows are tokens for x, y, dy and dx, and output
    features for w and dw (one scale per output channel, as each token
    carries one scale per activation row);
  * tensors are bf16; each product is the exact float64 product of the bf16
    operands rounded once to bf16 (wgrad.bf16_rne), the result an fp32
    accumulation rounds to whenever its sums are exact;
  * the dw_q that the optimiser receives is the unit's gradient, the one the
    controller takes the norm of.
"""
from __future__ import annotations

import numpy as np

from .fakequant import fakequant_rows
from .wgrad import bf16_rne, widen_bf16


def matmul_bf16(a_bits: np.ndarray, b_bits: np.ndarray) -> np.ndarray:
    """bf16(a b) for bf16 matrices a [r, k] and b [k, c] (uint16 bits): the
    exact float64 product (every term and sum exact for the operand sizes
    used here) rounded once to bf16."""
    return bf16_rne(widen_bf16(a_bits) @ widen_bf16(b_bits))


def forward(x_bits: np.ndarray, w_bits: np.ndarray, fmt: int) -> dict:
    """x [tokens, in], w [out, in] as bf16 bits; fmt the forward format."""
    x_q = fakequant_rows(x_bits, fmt)
    w_q = fakequant_rows(w_bits, fmt)
    y = matmul_bf16(x_q, w_q.T)
    return {"x_q": x_q, "w_q": w_q, "y": y, "y_q": fakequant_rows(y, fmt)}


def backward(dy_bits: np.ndarray, x_q: np.ndarray, w_q: np.ndarray, fmt: int) -> dict:
    """dy [tokens, out] as bf16 bits, with the forward's x_q and w_q; fmt the
    backward format."""
    dy_q = fakequant_rows(dy_bits, fmt)
    dx = matmul_bf16(dy_q, w_q)
    dw = matmul_bf16(dy_q.T, x_q)
    return {"dy_q": dy_q, "dx": dx, "dx_q": fakequant_rows(dx, fmt), "dw": dw,
            "dw_q": fakequant_rows(dw, fmt)}


def formats(in_recovery: bool, low: tuple, recovery: tuple) -> tuple:
    """(forward format, backward format) of a unit: `recovery` when the unit
    is in A_t, else `low` (Alg. 2)."""
    return recovery if in_recovery else low
