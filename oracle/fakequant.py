"""Oracle of the recovery actuator: per-token fake quantisation of saved
activations -- TEST INFRASTRUCTURE ONLY (same rules as the rest of oracle/).

What it computes (App. E.2, quantisation-simulated operators; Sec. 5.1 and
App. E.4, token-wise low-bit quantisation of saved activations; the INT8
low-cost path of the LLaMA-2 13B fine-tuning test, Sec. 5.3 and App. E.3): for each
token (one row of a unit's [tokens, features] activation matrix), the values
are scaled into the representable range of the target format, rounded to the
nearest representable value, and rescaled to the original range.  The format
is chosen per unit by the controller's mask: the low-cost format when the unit
is on the low-cost path, the recovery format when it is in A_t.

Readings:
  * formats are the OCP 8-bit and MX sub-byte floating-point formats without
    inf/NaN: E2M1 (max 6), E3M2 (max 28), E4M3 (max 448), E5M2 (max 57344);
    format 0 is the identity (the BF16 path);
  * INT8 (format 5) is symmetric per-token integer quantisation, the grid
    {-127, ..., 127} (the code -128 is not used, so the grid is symmetric):
    fmax = 127, q = rint(y) with ties to the even integer, clamped to
    [-127, 127]; the rest of the recipe is the one of the float formats;
  * arithmetic is fp32 with round-to-nearest-even: amax = max |x| over the
    token, inv = fmax / amax and s = amax / fmax (one division each per
    token), y = x * inv, q = the representable value nearest to y (ties to
    the even significand; magnitudes beyond fmax clamp to fmax), output =
    bf16_rne(q * s), keeping the sign of x (also for -0 and values that
    round to zero); an all-zero token becomes +0;
  * inputs and outputs are bf16 (given here as uint16 bit patterns).
"""
from __future__ import annotations

import numpy as np

# format id -> (mantissa bits, minimum normal exponent, largest finite value)
FORMATS = {
    1: (1, 0, 6.0),          # E2M1, bias 1
    2: (2, -2, 28.0),        # E3M2, bias 3
    3: (3, -6, 448.0),       # E4M3, bias 7 (no inf; S.1111.111 is NaN, so 448 is max)
    4: (2, -14, 57344.0),    # E5M2, bias 15
}
# integer format id -> largest magnitude of the symmetric grid
INT_FORMATS = {5: 127.0}   # INT8
FORMAT_NAMES = {0: "bf16", 1: "e2m1", 2: "e3m2", 3: "e4m3", 4: "e5m2", 5: "int8"}


def fmax_of(fmt: int) -> float:
    """Largest magnitude of a format's grid."""
    return INT_FORMATS[fmt] if fmt in INT_FORMATS else FORMATS[fmt][2]


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def round_to_format(y: np.ndarray, fmt: int) -> np.ndarray:
    """Nearest representable value of the format to each fp32 y (ties to the
    even significand), saturating at the largest finite value."""
    mbits, emin, fmax = FORMATS[fmt]
    y = np.asarray(y, np.float32)
    a = np.abs(y).astype(np.float64)          # exact
    _, E = np.frexp(a)                          # a = m * 2^E, m in [0.5, 1)
    e = np.maximum(E.astype(np.float64) - 1.0, emin)   # binade exponent, floor(log2 a)
    step = np.exp2(e - mbits)
    q = np.rint(a / step) * step                # a / step is exact (power of two)
    q = np.minimum(q, fmax)
    return np.copysign(q, y).astype(np.float32)     # the sign of y is kept, -0 included


def round_to_int(y: np.ndarray, fmt: int) -> np.ndarray:
    """Nearest integer to each fp32 y (ties to even), clamped to the
    symmetric grid [-qmax, qmax]; the sign of y is kept, -0 included."""
    qmax = INT_FORMATS[fmt]
    y = np.asarray(y, np.float32)
    q = np.minimum(np.rint(np.abs(y).astype(np.float64)), qmax)
    return np.copysign(q, y).astype(np.float32)


def fakequant_rows(x_bits: np.ndarray, fmt: int) -> np.ndarray:
    """Fake-quantise every row of a [rows, cols] bf16 matrix (uint16 bits)."""
    x_bits = np.asarray(x_bits, np.uint16)
    if fmt == 0:
        return x_bits.copy()
    fmax = fmax_of(fmt)
    x = bf16_to_f32(x_bits)
    amax = np.max(np.abs(x), axis=1, keepdims=True).astype(np.float32)
    nz = amax > 0
    safe = np.where(nz, amax, np.float32(1.0))
    inv = (np.float32(fmax) / safe).astype(np.float32)        # fp32 division, RNE
    s = (safe / np.float32(fmax)).astype(np.float32)          # fp32 division, RNE
    y = (x * inv).astype(np.float32)                           # fp32 product, RNE
    q = round_to_int(y, fmt) if fmt in INT_FORMATS else round_to_format(y, fmt)
    out = (q * s).astype(np.float32)                           # fp32 product, RNE
    out = np.where(nz, out, np.float32(0.0))
    return f32_to_bf16(out)


def actuate(units, mask, fmt_lo: int, fmt_hi: int):
    """units: list of [rows, cols] bf16 activation matrices, one per unit;
    mask[b] = 1 selects the recovery format for unit b (Alg. 2 actuator)."""
    return [fakequant_rows(x, fmt_hi if m else fmt_lo) for x, m in zip(units, mask)]
