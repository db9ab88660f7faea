"""Plain CPU oracle of the GNMR controller pass (float64, NumPy).

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import or call this module.  The product
path (the HIP library and its Python binding) never does, and this module
imports nothing from it.

What it computes, per controller step t = 1, 2, ... (paper notation):

  norm    n_{b,t} = ||g_{b,t}||_2 over all parameters of unit b; a unit made
          of several tensors is the L2 norm of their concatenation
          (Sec. 2, local-gradient equation; Sec. 3.4, block as unit).
  GNMR    1 if t = 1 or A_{b,t-1} = 0, else n_{b,t} / (A_{b,t-1} + eps)
          (Alg. 1; GNMR definition of Sec. 3.1).
  D-GNMR  GNMR_{b,t} / (mean(Q_b) + eps) once Q_b holds delta values, else 1;
          Q_b holds the delta previous GNMR values, the current one excluded
          (Alg. 1; Delta-GNMR definition of Sec. 3.2).
  state   A_{b,t} = A_{b,t-1} + (n_{b,t} - A_{b,t-1}) / t, then push GNMR_{b,t}
          into Q_b and keep the newest delta values (Alg. 1).
  risk    R_{b,t} = max(GNMR_{b,t} / alpha_t, D-GNMR_{b,t} / beta_t)
          (Alg. 2; Sec. 3.3).
  pool    C_t = {b : R_{b,t} > 1} U {b : Lock_b > 0}, recoverable units only,
          Lock_b as left by step t-1 (Alg. 2; Sec. 3.3).
  select  A_t = Top_maxO(C_t; R): all of C_t when |C_t| <= maxO, else the
          maxO members with the largest R; maxO caps the active set, it is not
          a quota (Alg. 2; Sec. 3.4; App. E.5 matched-trigger setting).
  locks   b in A_t and R > 1 -> Lock_b = T_lock; b in A_t and R <= 1 ->
          Lock_b = max(Lock_b - 1, 0); b not in A_t -> Lock_b = 0 (Alg. 2).

Readings where the paper is silent:
  * Ties in Top_maxO are broken by the smaller unit index.
  * eps = 0 with a zero D-GNMR denominator gives D-GNMR = 1 (the same
    convention Alg. 1 uses for A = 0).
  * t is the global controller step; every step is an observation, n = 0
    included.
  * Non-finite n (outside the paper): GNMR = D-GNMR = R = +inf, A_b kept,
    1.0 pushed into Q_b, counted in n_nonfinite.  A gradient whose sum of
    squares reaches 2^128 (the end of the fp32 range the gradient pass
    accumulates in) has norm +inf.
  * Statistics: n_trig_gnmr = #{GNMR/alpha > 1}, n_trig_dgnmr =
    #{D-GNMR/beta > 1}, n_trig = #{R > 1}, all over recoverable units;
    hit_maxo = 1 when the ranked pool is non-empty and at least maxO large.

Policy variants (both off by default):
  * budget_mode = BUDGET_ADMITTED caps only the newly admitted units, as the
    budget-convention remark of App. C allows: the candidates already in
    A_{t-1} stay active, and Top_maxO ranks the other candidates
    (A_t = (C_t & A_{t-1}) U Top_maxO(C_t minus A_{t-1}; R)).
  * warmup_steps = W: for t <= W every recoverable unit takes the recovery
    path (the high-fidelity warm-up of App. E.6): C_t = A_t = B_rec and the
    lock rule of Alg. 2 is applied to it; GNMR state updates as usual.
  * budget_mode = BUDGET_STATIC: the ADAPT-style static baseline of App. E.4.
    Steps 1..W run every recoverable unit on the recovery path and record
    GNMR; at t = W + 1 the maxO recoverable units of largest mean GNMR over
    steps 1..W (ties: smaller index) become the recovery set for good; no
    locks.  Counters: n_cand is |B_rec| up to t = W + 1, then |A_t|.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

F32 = 0
BF16 = 1

# budget conventions (Sec. 3.4; the budget-convention remark of App. C)
BUDGET_ACTIVE = 0      # |A_t| <= maxO (canonical)
BUDGET_ADMITTED = 1    # |A_t minus A_{t-1}| <= maxO: only newly admitted units count
BUDGET_STATIC = 2      # ADAPT-style static set fixed after a profiling warm-up (App. E.4)


# --------------------------------------------------------------------------
# norm  (Sec. 2, local-gradient equation)
# --------------------------------------------------------------------------

def widen(values: np.ndarray, dtype: int) -> np.ndarray:
    """Exact widening to float64.  bf16 is given as uint16 bit patterns."""
    if dtype == F32:
        return np.asarray(values, dtype=np.float32).astype(np.float64)
    if dtype == BF16:
        bits = np.asarray(values, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype}")


def sumsq(segments, chunk: int = 1 << 22) -> float:
    """Sum of squares over a unit's segments, each a (values, dtype) pair.

    Every square of a widened bf16 or fp32 value is exact in float64; only
    the summation rounds."""
    s = 0.0
    for values, dtype in segments:
        values = np.asarray(values).reshape(-1)
        for lo in range(0, values.size, chunk):
            x = widen(values[lo:lo + chunk], dtype)
            s += float(np.dot(x, x))
    return s


# The gradient pass accumulates sums of squares in fp32, whose range ends at
# 2^128.  Reading (non-finite norms are outside the paper): a unit whose sum
# of squares reaches 2^128, i.e. whose norm is 2^64 or more, has a non-finite
# norm, +inf.  NaN stays NaN.
SUMSQ_LIMIT = 2.0 ** 128


def unit_norm(segments) -> float:
    ss = sumsq(segments)
    if ss >= SUMSQ_LIMIT:
        return math.inf
    return math.sqrt(ss)


# --------------------------------------------------------------------------
# controller state and one step  (Alg. 1 and Alg. 2)
# --------------------------------------------------------------------------

@dataclass
class StepResult:
    t: int
    norm: np.ndarray
    gnmr: np.ndarray
    dgnmr: np.ndarray
    risk: np.ndarray
    mask: np.ndarray      # uint8, 1 = recovery path this step (b in A_t)
    lock: np.ndarray      # int32, Lock_b after the step
    stats: dict


class Controller:
    """Per-unit GNMR state: step counter t, historical means A_b, recent
    GNMR queues Q_b (length <= delta), lock counters Lock_b."""

    def __init__(self, num_units: int, window: int, max_o: int, lock_len: int,
                 eps: float, recoverable=None, budget_mode: int = BUDGET_ACTIVE,
                 warmup_steps: int = 0):
        if num_units < 1 or window < 1 or max_o < 0 or lock_len < 0:
            raise ValueError("need num_units >= 1, window >= 1, max_o >= 0, lock_len >= 0")
        if budget_mode not in (BUDGET_ACTIVE, BUDGET_ADMITTED, BUDGET_STATIC) or warmup_steps < 0:
            raise ValueError("unknown budget_mode or negative warmup_steps")
        if budget_mode == BUDGET_STATIC and warmup_steps < 1:
            raise ValueError("the static baseline needs warmup_steps >= 1")
        if not (eps >= 0.0 and math.isfinite(eps)):
            raise ValueError("need finite eps >= 0")
        self.U = int(num_units)
        self.delta = int(window)
        self.max_o = int(max_o)
        self.lock_len = int(lock_len)
        self.eps = float(eps)
        if recoverable is None:
            self.rec = np.ones(self.U, dtype=bool)
        else:
            self.rec = np.asarray(recoverable).astype(bool).reshape(-1)
            if self.rec.size != self.U:
                raise ValueError("recoverable must have num_units entries")
        self.budget_mode = int(budget_mode)
        self.warmup_steps = int(warmup_steps)
        self.t = 0                                   # steps taken so far
        self.A = np.zeros(self.U)                    # historical means A_b
        self.Q: list[np.ndarray] = []                # oldest first, each [U]
        self.lock = np.zeros(self.U, dtype=np.int64)
        self.active = np.zeros(self.U, dtype=bool)   # A_{t-1}
        self.gsum = np.zeros(self.U)                 # sum of GNMR over the profiling steps

    # -- state snapshot -----------------------------------------------------
    def get_state(self) -> dict:
        return {"t": self.t, "A": self.A.copy(), "Q": [q.copy() for q in self.Q],
                "lock": self.lock.copy(), "active": self.active.copy(),
                "gsum": self.gsum.copy()}

    def set_state(self, st: dict) -> None:
        self.t = int(st["t"])
        self.A = np.array(st["A"], dtype=np.float64)
        self.Q = [np.array(q, dtype=np.float64) for q in st["Q"]]
        self.lock = np.array(st["lock"], dtype=np.int64)
        self.active = np.array(st["active"], dtype=bool)
        self.gsum = np.array(st["gsum"], dtype=np.float64)

    # -- one controller step --------------------------------------------------
    def step(self, norms, alpha: float, beta: float) -> StepResult:
        if not (alpha > 0 and beta > 0 and math.isfinite(alpha) and math.isfinite(beta)):
            raise ValueError("thresholds must be finite and > 0")
        n = np.asarray(norms, dtype=np.float64).reshape(-1)
        if n.size != self.U:
            raise ValueError("one norm per unit expected")
        U, delta, eps = self.U, self.delta, self.eps
        t = self.t + 1
        finite = np.isfinite(n)

        # Alg. 1: GNMR = 1 at t = 1 or when the historical mean is 0.
        gnmr = np.ones(U)
        if t > 1:
            has_mean = finite & (self.A != 0.0)
            gnmr[has_mean] = n[has_mean] / (self.A[has_mean] + eps)

        # Alg. 1: Delta-GNMR against the mean of the delta previous GNMRs.
        dgnmr = np.ones(U)
        if len(self.Q) == delta:
            total = np.zeros(U)
            for q in self.Q:                       # oldest to newest
                total = total + q
            den = total / delta + eps
            ok = finite & (den != 0.0)
            dgnmr[ok] = gnmr[ok] / den[ok]

        # Alg. 1: running mean and queue push.
        A_next = self.A + (n - self.A) / t
        self.A = np.where(finite, A_next, self.A)
        pushed = np.where(finite, gnmr, 1.0)
        self.Q.append(pushed)
        if len(self.Q) > delta:
            self.Q.pop(0)

        gnmr = np.where(finite, gnmr, np.inf)
        dgnmr = np.where(finite, dgnmr, np.inf)

        # Alg. 2: combined risk.
        g_term = gnmr / alpha
        d_term = dgnmr / beta
        risk = np.maximum(g_term, d_term)

        # Alg. 2: candidate pool (lock counters from the previous step).
        triggered = self.rec & (risk > 1.0)
        cand = triggered | (self.rec & (self.lock > 0))
        if self.budget_mode == BUDGET_STATIC:
            return self._static_step(t, n, gnmr, dgnmr, risk, g_term, d_term, triggered, finite)
        warm = t <= self.warmup_steps
        if warm:
            # high-fidelity warm-up (App. E.6): every recoverable unit recovers
            cand = self.rec.copy()
        cand_idx = np.flatnonzero(cand)

        # Units that skip the ranking: all of them during the warm-up; under the
        # admitted-only budget, the candidates already active at t-1.
        if warm:
            keep = cand
        elif self.budget_mode == BUDGET_ADMITTED:
            keep = cand & self.active
        else:
            keep = np.zeros(U, dtype=bool)
        pool_idx = np.flatnonzero(cand & ~keep)

        # Alg. 2: Top_maxO by R, ties to the smaller index.
        if pool_idx.size <= self.max_o:
            admitted = pool_idx
        else:
            order = np.lexsort((pool_idx, -risk[pool_idx]))
            admitted = pool_idx[order[: self.max_o]]
        active = np.union1d(np.flatnonzero(keep), admitted).astype(np.int64)
        mask = np.zeros(U, dtype=np.uint8)
        mask[active] = 1

        # Alg. 2: lock update.
        new_lock = np.zeros(U, dtype=np.int64)
        for b in active:
            if risk[b] > 1.0:
                new_lock[b] = self.lock_len
            else:
                new_lock[b] = max(self.lock[b] - 1, 0)
        self.lock = new_lock
        self.active = mask.astype(bool)
        self.t = t

        stats = {
            "t": t,
            "n_trig_gnmr": int(np.count_nonzero(self.rec & (g_term > 1.0))),
            "n_trig_dgnmr": int(np.count_nonzero(self.rec & (d_term > 1.0))),
            "n_trig": int(np.count_nonzero(triggered)),
            "n_cand": int(cand_idx.size),
            "n_active": int(active.size),
            "hit_maxo": int(not warm and pool_idx.size > 0 and pool_idx.size >= self.max_o),
            "n_nonfinite": int(np.count_nonzero(~finite)),
        }
        return StepResult(t, n.copy(), gnmr, dgnmr, risk, mask,
                          self.lock.astype(np.int32), stats)


    def _static_step(self, t, n, gnmr, dgnmr, risk, g_term, d_term, triggered, finite):
        """ADAPT-style static baseline (App. E.4): for t <= W every recoverable
        unit takes the recovery path while sum(GNMR) is recorded; at t = W + 1
        the maxO recoverable units with the largest mean GNMR over steps 1..W
        (ties: smaller index) become the recovery set, fixed from then on.
        Locks are not used."""
        U, W = self.U, self.warmup_steps
        ranked = np.zeros(0, dtype=np.int64)
        if t <= W:
            self.gsum = self.gsum + np.where(finite, gnmr, 0.0)
            active = np.flatnonzero(self.rec)
        elif t == W + 1:
            mean = self.gsum / W
            ranked = np.flatnonzero(self.rec)
            order = np.lexsort((ranked, -mean[ranked]))
            active = np.sort(ranked[order[: self.max_o]])
        else:
            active = np.flatnonzero(self.active)
        mask = np.zeros(U, dtype=np.uint8)
        mask[active] = 1
        self.active = mask.astype(bool)
        self.lock = np.zeros(U, dtype=np.int64)
        self.t = t
        stats = {
            "t": t,
            "n_trig_gnmr": int(np.count_nonzero(self.rec & (g_term > 1.0))),
            "n_trig_dgnmr": int(np.count_nonzero(self.rec & (d_term > 1.0))),
            "n_trig": int(np.count_nonzero(triggered)),
            "n_cand": int(np.count_nonzero(self.rec)) if t <= W + 1 else int(active.size),
            "n_active": int(active.size),
            "hit_maxo": int(ranked.size > 0 and ranked.size >= self.max_o),
            "n_nonfinite": int(np.count_nonzero(~finite)),
        }
        return StepResult(t, n.copy(), gnmr, dgnmr, risk, mask, self.lock.astype(np.int32),
                          stats)
