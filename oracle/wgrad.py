"""Oracle of the producer-fused gradient pass -- TEST INFRASTRUCTURE ONLY
(same rules as the rest of oracle/: only tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline leg may use it; it imports nothing from the HIP
library or its binding).

What it computes.  A recoverable unit here is the weight of a linear layer
y = x W^T (the operator view of Sec. 2).  Its gradient over a batch of
tokens is dW = dy^T x, i.e. dW[o][i] = sum_t dy[t][o] * x[t][i], and the
controller needs the L2 norm of that gradient (Sec. 2, local-gradient
equation; Alg. 1).  The gradient is stored in bf16, so the norm the
controller sees is the norm of the stored bf16 values; it is split here into
the sums of squares over the 256x256 tiles of dW, in row-major tile order,
which is the unit of work of the fused kernel.

Readings:
  * stored gradient = bf16 round-to-nearest-even of the product;
  * the exact product is the float64 matrix product of the exactly widened
    bf16 operands; for the operand sizes used here (at most a few thousand
    tokens of values below 2^8 in magnitude after scaling) every product is
    exact in float64 and the float64 sum carries a relative error of at most
    tokens * 2^-53 of sum |dy| |x|, far below the bounds checked against;
  * the fused kernel accumulates in fp32 (matrix cores), in an order it
    chooses, then rounds once to bf16.  error_bound() is the bound such a
    result obeys: |q - exact| <= 2^-8 (|exact| + g S) + g S, S = |dy|^T |x|,
    g = K u / (1 - K u) with u = 2^-23 (one unit of fp32 precision per
    addition, which also covers directed rounding inside the accumulator),
    plus 2^-133 for bf16 underflow;
  * gradient accumulation over micro-batches: the kernel adds its fp32
    accumulation to the stored bf16 gradient in fp32 (one rounding) and
    rounds the sum to bf16 once; error_bound_accumulate() states the bound.
"""
from __future__ import annotations

import numpy as np

TILE = 256


def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64, exactly."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def wgrad_exact(dy_bits: np.ndarray, x_bits: np.ndarray) -> np.ndarray:
    """dW = dy^T x in float64; dy [tokens][out], x [tokens][in] as bf16 bits."""
    dy = widen_bf16(dy_bits)
    x = widen_bf16(x_bits)
    assert dy.ndim == 2 and x.ndim == 2 and dy.shape[0] == x.shape[0]
    return dy.T @ x


def bf16_rne(v: np.ndarray) -> np.ndarray:
    """Correctly rounded float64 -> bf16 (round to nearest, ties to even),
    one rounding, as uint16 bit patterns.  Overflow gives +-inf, NaN a quiet
    NaN.  With a = m 2^e (0.5 <= m < 1) the bf16 spacing at a is 2^(e-8)
    (8 significant bits), or 2^-133 below the smallest normal; a / spacing
    is exact and rint rounds half to even."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    finite = np.isfinite(a)
    af = np.where(finite, a, 0.0)
    _, e = np.frexp(af)
    e = np.maximum(e, -125)
    spacing = np.exp2((e - 8).astype(np.float64))
    q = np.rint(af / spacing) * spacing
    largest = (2.0 - 2.0 ** -7) * 2.0 ** 127
    over = (q > largest) | np.isinf(a)
    q = np.where(over, 0.0, q)
    bits = (q.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    bits = np.where(over, np.uint16(0x7F80), bits)
    bits = np.where(np.signbit(v), bits | np.uint16(0x8000), bits)
    return np.where(np.isnan(v), np.uint16(0x7FC0), bits).astype(np.uint16)


def tile_sumsq(dw_bits: np.ndarray, tile: int = TILE) -> np.ndarray:
    """float64 sum of squares of the bf16 values over each tile x tile block
    of dW ([out][in]), in row-major tile order; edge tiles hold what is left."""
    w = widen_bf16(dw_bits)
    M, N = w.shape
    tm, tn = -(-M // tile), -(-N // tile)
    out = np.zeros(tm * tn, dtype=np.float64)
    for a in range(tm):
        for b in range(tn):
            blk = w[a * tile:(a + 1) * tile, b * tile:(b + 1) * tile]
            out[a * tn + b] = float(np.sum(blk * blk))
    return out


def num_tiles(out_features: int, in_features: int, tile: int = TILE) -> int:
    return (-(-out_features // tile)) * (-(-in_features // tile))


def error_bound(dy_bits: np.ndarray, x_bits: np.ndarray, exact: np.ndarray) -> np.ndarray:
    """Elementwise bound on |q - exact| for q = bf16(fp32 accumulation)."""
    K = np.asarray(dy_bits).shape[0]
    u = 2.0 ** -23
    g = K * u / (1.0 - K * u) if K > 0 else 0.0
    S = np.abs(widen_bf16(dy_bits)).T @ np.abs(widen_bf16(x_bits))
    return 2.0 ** -8 * (np.abs(exact) + g * S) + g * S + 2.0 ** -133


def wgrad_accumulate_exact(old_bits: np.ndarray, dy_bits: np.ndarray,
                           x_bits: np.ndarray) -> np.ndarray:
    """Gradient accumulation over micro-batches: the stored bf16 gradient
    plus this micro-batch's dW = dy^T x, in float64 (exact for the operand
    sizes used here, as in wgrad_exact)."""
    return widen_bf16(old_bits) + wgrad_exact(dy_bits, x_bits)


def error_bound_accumulate(old_bits: np.ndarray, dy_bits: np.ndarray, x_bits: np.ndarray,
                           exact: np.ndarray) -> np.ndarray:
    """Elementwise bound on |q - exact| for q = bf16(fp32(old + a)), a the
    fp32 accumulation of the product P: with |a - P| <= g S (as in
    error_bound), z = fp32(old + a) is within 2^-24 |old + a| of old + a, and
    bf16(z) within 2^-8 |z| of z (a full bf16 unit, twice the RNE bound, as
    in error_bound), so with |old + a| <= |exact| + g S:
    |q - exact| <= g S + (|exact| + g S) (2^-8 (1 + 2^-24) + 2^-24)
               <  g S + (|exact| + g S) (2^-8 + 2^-22), plus 2^-133 for bf16
    underflow."""
    K = np.asarray(dy_bits).shape[0]
    u = 2.0 ** -23
    g = K * u / (1.0 - K * u) if K > 0 else 0.0
    S = np.abs(widen_bf16(dy_bits)).T @ np.abs(widen_bf16(x_bits))
    return g * S + (np.abs(exact) + g * S) * (2.0 ** -8 + 2.0 ** -22) + 2.0 ** -133


def unit_norm(dw_bits: np.ndarray) -> float:
    """L2 norm of a unit's stored bf16 gradient (float64)."""
    w = widen_bf16(dw_bits)
    return float(np.sqrt(np.sum(w * w)))
