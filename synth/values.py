"""Counter-based synthetic gradient values (host twin, NumPy).

Every gradient element is a pure function of ``(seed, t, b, i)`` -- seed,
controller step, unit index, element index inside the unit's concatenated
segments -- and of the fp32 scale ``s[b, t]``:

    key(seed, t, b) = mix64(mix64(c + GAMMA) + GAMMA),
        c = (seed << 48) | (t << 24) | b          (seed < 2^16, t, b < 2^24)
    h(i)            = mix64(key + (i // 4 + 1) * GAMMA)          (mod 2^64)
    j(i)            = (h(i) >> (16 * (i % 4))) & 0xFFFF
    x(i)            = rnd_dtype( s * Z[j(i)] )     (one IEEE fp32 multiply)

``mix64`` is the output finaliser of SplitMix64 (Steele, Lea and Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014) and GAMMA its
golden-ratio increment, so ``h`` is the SplitMix64 sequence seeded with
``key``.  ``Z`` is a 2^16-entry fp32 table of standard-normal quantiles
Z[j] = Phi^-1((j + 1/2) / 2^16), computed once in float64 with
``scipy.special.ndtri`` and rounded to fp32.  ``rnd_bf16`` is
round-to-nearest-even on the fp32 bit pattern; for fp32 it is the identity.

Only integer steps, one table lookup and one fp32 multiply are involved, so
the HIP generator kernel (synth/csrc/gen.hip) reproduces these values bit for
bit.  Nothing here computes any part of the controller.
"""
from __future__ import annotations

import functools

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MUL1 = 0xBF58476D1CE4E5B9
MUL2 = 0x94D049BB133111EB
TABLE_BITS = 16

DTYPE_F32 = 0
DTYPE_BF16 = 1
DTYPE_NAMES = {DTYPE_F32: "f32", DTYPE_BF16: "bf16"}
DTYPE_SIZE = {DTYPE_F32: 4, DTYPE_BF16: 2}


def mix64_int(z: int) -> int:
    """SplitMix64 finaliser on a Python int (exact, mod 2^64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MUL1) & MASK64
    z = ((z ^ (z >> 27)) * MUL2) & MASK64
    return z ^ (z >> 31)


def mix64_np(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser on a uint64 array (NumPy integer ops wrap mod 2^64).
    Works in place on z and returns it."""
    t = z >> np.uint64(30)
    z ^= t
    z *= np.uint64(MUL1)
    np.right_shift(z, np.uint64(27), out=t)
    z ^= t
    z *= np.uint64(MUL2)
    np.right_shift(z, np.uint64(31), out=t)
    z ^= t
    return z


def unit_key(seed: int, t: int, b: int) -> int:
    if not (0 <= seed < (1 << 16) and 0 <= t < (1 << 24) and 0 <= b < (1 << 24)):
        raise ValueError(f"counter fields out of range: seed={seed} t={t} b={b}")
    c = (seed << 48) | (t << 24) | b
    return mix64_int(mix64_int(c + GAMMA) + GAMMA)


@functools.lru_cache(maxsize=1)
def normal_table() -> np.ndarray:
    """fp32 table of Phi^-1((j + 0.5) / 2^16), j = 0 .. 2^16 - 1."""
    from scipy.special import ndtri

    n = 1 << TABLE_BITS
    p = (np.arange(n, dtype=np.float64) + 0.5) / n
    tab = ndtri(p).astype(np.float32)
    tab.setflags(write=False)
    return tab


def table_indices(seed: int, t: int, b: int, start: int, count: int) -> np.ndarray:
    """16-bit table indices j(i) for unit elements i in [start, start + count).

    One 64-bit hash serves the four elements 4g .. 4g+3; field i % 4 is the
    (i % 4)-th 16-bit word of the hash, i.e. the little-endian uint16 view."""
    if count <= 0:
        return np.zeros(0, dtype=np.uint16)
    g0, g1 = start >> 2, (start + count + 3) >> 2
    key = np.uint64(unit_key(seed, t, b))
    h = np.arange(g0 + 1, g1 + 1, dtype=np.uint64)
    h *= np.uint64(GAMMA)
    h += key
    words = mix64_np(h).astype("<u8", copy=False).view("<u2")
    off = start - 4 * g0
    return words[off:off + count]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, returned as uint16 bit patterns.

    Inputs are finite (the generator never makes inf/NaN)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def unit_values(seed: int, t: int, b: int, scale: float, dtype: int,
                start: int, count: int, chunk: int = 1 << 22) -> np.ndarray:
    """Elements [start, start+count) of unit b at step t.

    Returns float32 values for DTYPE_F32 and uint16 bf16 bit patterns for
    DTYPE_BF16 (NumPy has no bfloat16)."""
    if dtype not in (DTYPE_F32, DTYPE_BF16):
        raise ValueError(f"unknown dtype {dtype}")
    s = np.float32(scale)
    tab = normal_table()
    out = np.empty(max(count, 0), dtype=np.float32 if dtype == DTYPE_F32 else np.uint16)
    for lo in range(0, max(count, 0), chunk):
        n = min(chunk, count - lo)
        x = tab[table_indices(seed, t, b, start + lo, n)]
        x *= s                       # one IEEE fp32 multiply, round to nearest even
        out[lo:lo + n] = x if dtype == DTYPE_F32 else f32_to_bf16_bits(x)
    return out
