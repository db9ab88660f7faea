"""Seeded operands for the weight-gradient GEMM: the output gradient dy
[tokens][out] and the layer input x [tokens][in] of a linear layer, as bf16
bit patterns.  Shared by the oracle side and the device side of the tests
and the benchmark; computes nothing of the method.

Values come from the counter-based generator of synth.values (its plain-C
twin): dy of unit b is the generator's unit 2*(b + BASE), x its unit
2*(b + BASE) + 1, at controller step t, with fp32 scales dy_scale and
x_scale.  Spikes are injected as a larger dy_scale, exactly as the gradient
workloads inject them.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import host
from . import values as V

BASE = 1 << 20   # generator unit ids above every gradient workload's units

# one LLaMA-2-13B decoder layer: q, k, v, o (5120x5120), gate, up (13824x5120),
# down (5120x13824), as [out_features, in_features]
LLAMA2_13B_LAYER = ((5120, 5120), (5120, 5120), (5120, 5120), (5120, 5120),
                    (13824, 5120), (13824, 5120), (5120, 13824))


def operands(seed: int, t: int, b: int, tokens: int, out_f: int, in_f: int,
             dy_scale: float = 1e-3, x_scale: float = 1.0):
    """(dy, x) bf16 bit arrays of shapes [tokens, out_f] and [tokens, in_f]."""
    u = 2 * (b + BASE)
    dy = host.unit_values(seed, t, u, np.float32(dy_scale), V.DTYPE_BF16, 0, tokens * out_f)
    x = host.unit_values(seed, t, u + 1, np.float32(x_scale), V.DTYPE_BF16, 0, tokens * in_f)
    return dy.reshape(tokens, out_f), x.reshape(tokens, in_f)


def small_integer_operands(seed: int, tokens: int, out_f: int, in_f: int, vmax: int = 1):
    """(dy, x) with integer values in [-vmax, vmax] (exact in bf16), for cases
    where every partial sum is an integer of at most tokens * vmax^2 in
    magnitude, so fp32 accumulation and the final bf16 rounding are exact
    while tokens * vmax^2 <= 256."""
    rng = np.random.default_rng(seed)
    def bits(shape):
        v = rng.integers(-vmax, vmax + 1, size=shape).astype(np.float32)
        return (v.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return bits((tokens, out_f)), bits((tokens, in_f))


@dataclass(frozen=True)
class WgradLayer:
    """The weight-gradient GEMMs of one decoder layer at `tokens` tokens."""
    name: str
    shapes: tuple
    tokens: int
    seed: int = 0

    @property
    def num_units(self) -> int:
        return len(self.shapes)

    @property
    def flops(self) -> int:
        return sum(2 * self.tokens * o * i for o, i in self.shapes)

    @property
    def grad_bytes(self) -> int:
        return sum(2 * o * i for o, i in self.shapes)

    @property
    def operand_bytes(self) -> int:
        """dy and x of every GEMM, bf16, each read once."""
        return sum(2 * self.tokens * (o + i) for o, i in self.shapes)

    def dy_scale(self, t: int, b: int) -> float:
        """Per-unit output-gradient scale: LogUniform[1e-4, 1e-2] per unit
        (drawn once from the seed), x10 in unit (t mod 7) at every step t
        that is a multiple of 4 (a spike the controller must catch)."""
        rng = np.random.default_rng([self.seed, 0x5767])
        sig = np.exp(rng.uniform(np.log(1e-4), np.log(1e-2), size=self.num_units))
        k = 10.0 if (t % 4 == 0 and b == t % self.num_units) else 1.0
        return float(np.float32(sig[b] * k))


def llama2_13b_layer(tokens: int = 4096) -> WgradLayer:
    return WgradLayer("llama2-13b-layer-wgrad", LLAMA2_13B_LAYER, tokens)
