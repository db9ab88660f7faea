"""Host-side threshold schedule (the per-step alpha_t, beta_t arguments)."""
import math


def two_stage_alpha(t: int, steps: int, hi: float = 1.5, lo: float = 1.1,
                    frac: float = 0.025) -> float:
    """Two-stage GNMR threshold: `hi` for the first ceil(frac * steps) steps (at
    least one), `lo` afterwards (Sec. 3.4 calibration; the recipe-level and
    13B fine-tuning settings use 1.5 -> 1.1 over the first 2.5% of steps)."""
    return hi if t <= max(1, math.ceil(frac * steps)) else lo
