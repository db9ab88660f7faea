"""Seeded synthetic workloads shaped like the paper's gradient sets.

A workload is a list of recoverable units (one linear weight matrix, or a
row block of one, per unit), a stream length T, the controller settings
(budget maxO, lock length T_lock, window delta, epsilon) and a table of
per-unit, per-step fp32 scales ``s[t, b]``.  Gradient elements are then
``s[t, b] * z`` with ``z`` from the counter-based normal table in
``synth.values``.

The unit lists follow the operator-level view of a transformer block
(Sec. 2 and App. B): per layer the attention projections q, k, v, o and the
SwiGLU projections gate, up, down, each a monitored and recoverable unit;
the MoE set adds per-expert gate/up/down units.  Stream structure (per-unit
scale, injected k-fold spikes, routing masks, drifting scales) is synthetic:
no gradient stream of the paper is available, these stand in for them.

Nothing here computes any part of the controller.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .values import DTYPE_BF16, DTYPE_F32, DTYPE_SIZE


@dataclass(frozen=True)
class Unit:
    name: str
    numel: int
    dtype: int
    pieces: tuple = ()      # segment lengths when the unit owns several tensors


@dataclass
class Workload:
    name: str
    units: list
    steps: int
    max_o: int
    lock_len: int
    window: int = 5
    eps: float = 1e-12
    seed: int = 0
    # scale[t-1, b] in float64 before rounding to fp32 (t = 1..steps)
    scale64: np.ndarray = field(repr=False, default=None)
    description: str = ""

    @property
    def num_units(self) -> int:
        return len(self.units)

    @property
    def numel(self) -> np.ndarray:
        return np.array([u.numel for u in self.units], dtype=np.int64)

    @property
    def dtypes(self) -> np.ndarray:
        return np.array([u.dtype for u in self.units], dtype=np.int32)

    @property
    def bytes_per_step(self) -> int:
        return int(sum(u.numel * DTYPE_SIZE[u.dtype] for u in self.units))

    def scale32(self, t: int, nudge: np.ndarray | None = None) -> np.ndarray:
        """fp32 scales of step t (1-based), optionally times a per-unit nudge
        factor; the product is formed in float64 and rounded once."""
        s = self.scale64[t - 1]
        if nudge is not None:
            s = s * nudge
        return s.astype(np.float32)

    def alpha(self, t: int) -> float:
        return two_stage_alpha(t, self.steps)

    def beta(self, t: int) -> float:
        return 1.5


def two_stage_alpha(t: int, steps: int, hi: float = 1.5, lo: float = 1.1,
                    frac: float = 0.025) -> float:
    """Two-stage GNMR threshold: ``hi`` for the first ceil(frac * steps) steps
    (at least one), ``lo`` afterwards (Sec. 3.4 calibration; App. E.2 recipe
    and 13B fine-tuning setting: 1.5 -> 1.1, first 2.5% of steps)."""
    return hi if t <= max(1, math.ceil(frac * steps)) else lo


def _log_uniform(rng, lo, hi, size=None):
    return np.exp(rng.uniform(math.log(lo), math.log(hi), size=size))


def dense_units(layers: int, d: int, ffn: int, dtype: int, row_block: int = 0) -> list:
    """q, k, v, o ([d, d]), gate, up ([ffn, d]) and down ([d, ffn]) per layer,
    row-major [out, in].  With row_block > 0 each matrix is split into blocks
    of row_block rows (the last block may be shorter), each its own unit."""
    mats = [("q", d, d), ("k", d, d), ("v", d, d), ("o", d, d),
            ("gate", ffn, d), ("up", ffn, d), ("down", d, ffn)]
    units = []
    for layer in range(layers):
        for name, rows, cols in mats:
            if row_block <= 0:
                units.append(Unit(f"L{layer}.{name}", rows * cols, dtype))
            else:
                for r0 in range(0, rows, row_block):
                    r = min(row_block, rows - r0)
                    units.append(Unit(f"L{layer}.{name}[{r0}:{r0 + r}]", r * cols, dtype))
    return units


def layer_units(layers: int, d: int, ffn: int, dtype: int) -> list:
    """Block-as-unit (Sec. 3.4): each decoder layer is one unit owning its
    seven projection weights as seven segments (q, k, v, o, gate, up, down)."""
    pieces = (d * d,) * 4 + (ffn * d,) * 2 + (d * ffn,)
    return [Unit(f"L{layer}", sum(pieces), dtype, pieces) for layer in range(layers)]


def moe_units(layers: int = 27, hidden: int = 2048, expert_ffn: int = 1408,
              routed: int = 64, shared: int = 2, dtype: int = DTYPE_F32) -> list:
    units = []
    for layer in range(layers):
        for name in ("q", "k", "v", "o"):
            units.append(Unit(f"L{layer}.attn.{name}", hidden * hidden, dtype))
        for kind, count in (("shared", shared), ("routed", routed)):
            for e in range(count):
                for name in ("gate", "up", "down"):
                    units.append(Unit(f"L{layer}.{kind}{e}.{name}", expert_ffn * hidden, dtype))
    return units


def _spiky_stream(units, steps, seed, spike_steps, units_per_spike, k_choices,
                  every_step=False):
    """sigma_b ~ LogUniform[1e-4, 1e-2]; k-fold spikes on chosen unit-steps."""
    rng = np.random.Generator(np.random.PCG64(seed))
    U = len(units)
    sigma = _log_uniform(rng, 1e-4, 1e-2, size=U)
    k = np.ones((steps, U))
    if every_step:
        chosen_steps = list(range(1, steps + 1))
    else:
        chosen_steps = sorted(rng.choice(np.arange(2, steps + 1), size=spike_steps, replace=False).tolist())
    for t in chosen_steps:
        bs = rng.choice(U, size=units_per_spike, replace=False)
        for b in bs:
            k[t - 1, b] = float(rng.choice(k_choices))
    return sigma[None, :] * k, chosen_steps


def tiny(seed: int = 0) -> Workload:
    units = dense_units(4, 256, 688, DTYPE_F32)
    scale, spikes = _spiky_stream(units, 64, seed, 3, 2, [20.0])
    return Workload("tiny", units, 64, max_o=2, lock_len=4, seed=seed, scale64=scale,
                    description="4-layer transformer, d=256, ffn=688, 28 fp32 units, "
                                f"x20 spikes at steps {spikes}")


def llama7b(seed: int = 0) -> Workload:
    units = dense_units(32, 4096, 11008, DTYPE_BF16)
    scale, spikes = _spiky_stream(units, 16, seed, 3, 2, [20.0])
    return Workload("llama2-7b", units, 16, max_o=8, lock_len=8, seed=seed, scale64=scale,
                    description="LLaMA-2-7B-shaped, 224 bf16 units, "
                                f"x20 spikes at steps {spikes}")


def llama13b(seed: int = 0) -> Workload:
    units = dense_units(40, 5120, 13824, DTYPE_BF16)
    per_step = int(round(0.01 * len(units)))
    scale, _ = _spiky_stream(units, 16, seed, 0, per_step, [10.0, 50.0], every_step=True)
    return Workload("llama2-13b", units, 16, max_o=8, lock_len=8, seed=seed, scale64=scale,
                    description="LLaMA-2-13B-shaped, 280 bf16 units, x10/x50 spikes "
                                f"in {per_step} units every step")


def llama13b_layers(seed: int = 0) -> Workload:
    """The paper's 13B controller setting: maxO = 10 over 40 decoder layers,
    T_lock = 1, two-stage alpha 1.5 -> 1.1, beta = 1.5, window 5 (App. E.3),
    on the LLaMA-2-13B-shaped bf16 gradient set with each layer one unit."""
    units = layer_units(40, 5120, 13824, DTYPE_BF16)
    scale, _ = _spiky_stream(units, 16, seed, 0, 1, [10.0, 50.0], every_step=True)
    return Workload("llama2-13b-layers", units, 16, max_o=10, lock_len=1, seed=seed,
                    scale64=scale,
                    description="LLaMA-2-13B-shaped, 40 block units of 7 bf16 segments, "
                                "x10/x50 spike in one layer every step")


def moe(seed: int = 0) -> Workload:
    units = moe_units()
    steps = 32
    rng = np.random.Generator(np.random.PCG64(seed))
    U = len(units)
    sigma = _log_uniform(rng, 1e-4, 1e-2, size=U)
    m = np.ones((steps, U))
    per_layer = 4 + (2 + 64) * 3
    for layer in range(27):
        base = layer * per_layer + 4 + 2 * 3
        routed_off = rng.random((steps, 64)) < 0.7  # expert not routed this step
        for e in range(64):
            for j in range(3):
                m[:, base + 3 * e + j] = np.where(routed_off[:, e], 0.0, 1.0)
    return Workload("moe", units, steps, max_o=32, lock_len=4, seed=seed,
                    scale64=sigma[None, :] * m,
                    description="DeepSeek-style MoE, 27 layers, 64 routed + 2 shared experts "
                                "(gate/up/down units) + 4 attention units, fp32, routed "
                                "experts zero-masked with p=0.7 per step")


def fine(seed: int = 0, row_block: int = 128) -> Workload:
    units = dense_units(32, 4096, 11008, DTYPE_BF16, row_block=row_block)
    steps = 256
    rng = np.random.Generator(np.random.PCG64(seed))
    U = len(units)
    log_s0 = np.log(_log_uniform(rng, 1e-4, 1e-2, size=U))
    walk = np.cumsum(rng.normal(0.0, 0.01, size=(steps, U)), axis=0)
    k = np.ones((steps, U))
    starts = sorted(rng.choice(np.arange(2, steps), size=8, replace=False).tolist())
    per_burst = int(round(0.01 * U))
    for t0 in starts:
        bs = rng.choice(U, size=per_burst, replace=False)
        kk = _log_uniform(rng, 5.0, 50.0, size=per_burst)
        for t in (t0, t0 + 1):
            k[t - 1, bs] *= kk
    scale = np.exp(log_s0[None, :] + walk) * k
    return Workload(f"fine{row_block}", units, steps, max_o=64, lock_len=16, seed=seed,
                    scale64=scale,
                    description=f"LLaMA-2-7B shape split into {row_block}-row blocks "
                                f"({U} bf16 units), log-std random walk, bursts at {starts}")


WORKLOADS = {
    "tiny": tiny,
    "llama2-7b": llama7b,
    "llama2-13b": llama13b,
    "llama2-13b-layers": llama13b_layers,
    "moe": moe,
    "fine128": lambda seed=0: fine(seed, 128),
    "fine32": lambda seed=0: fine(seed, 32),
}


def get(name: str, seed: int = 0) -> Workload:
    return WORKLOADS[name](seed)


def surrogate_norms(w: Workload, seed: int = 1) -> np.ndarray:
    """Norm-level stand-in for the gradient stream: n[t, b] =
    s[t, b] * sqrt(N_b) * (1 + xi / sqrt(2 N_b)), xi ~ N(0, 1), which is the
    scale and the relative spread of ||s z|| for N_b iid standard normals.
    float64, shape [steps, U]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    N = w.numel.astype(np.float64)
    xi = rng.normal(size=w.scale64.shape)
    return w.scale64 * np.sqrt(N)[None, :] * (1.0 + xi / np.sqrt(2.0 * N)[None, :])
