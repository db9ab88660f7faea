"""Test-side drivers: oracle norms of synthetic gradients, and the guard
co-simulation that keeps every decision of a stream away from its threshold.

The GPU accumulates squares in fp32 and the oracle in fp64, so their norms
differ by about 1e-6 relative.  A mask can only be compared bit for bit when
no decision sits within that distance of its threshold.  On oracle values,
every step must satisfy
  (G1) |GNMR/alpha - 1| > 1e-4, and |D-GNMR/beta - 1| > 1e-4 once the window
       is full, for every recoverable unit;
  (G2) when the ranked pool (C_t; C_t minus A_{t-1} under the admitted-only
       budget; none in a warm-up step) holds more than maxO units, the
       maxO-th and (maxO+1)-th largest R are either at least 1e-4 apart
       relative, or exactly equal (a tie both sides compute identically, e.g.
       the clamped value 1/beta) with the nearest distinct R above and below
       the tied value at least 1e-4 away from it (so that no unit can move
       across the tied group).
A unit-step that breaks either is nudged: its fp32 scale is multiplied by
(1 + 3e-4 j) for j = 1, -1, 2, -2, ... and the step is recomputed.
"""
from __future__ import annotations

import numpy as np

from oracle import BUDGET_ACTIVE, BUDGET_ADMITTED, Controller, unit_norm
from synth import values as V

GUARD = 1e-4


def host_unit_norm(seed, t, b, scale32, dtype, numel, pieces=None):
    """Oracle norm of unit b at step t from host-generated values."""
    if pieces is None:
        pieces = [numel]
    segs, start = [], 0
    for n in pieces:
        segs.append((V.unit_values(seed, t, b, float(scale32), dtype, start, n), dtype))
        start += n
    return unit_norm(segs)


def host_norms(w, t, scale32, units=None):
    sel = range(w.num_units) if units is None else units
    out = {}
    for b in sel:
        u = w.units[b]
        out[b] = host_unit_norm(w.seed, t, b, scale32[b], u.dtype, u.numel)
    return out


def violations(res, alpha, beta, max_o, window_full, lock_before, rec=None,
               active_before=None, warm=False):
    """Units whose decisions break G1 or G2 at this step (oracle values).
    active_before: A_{t-1} when the admitted-only budget ranks only the new
    candidates; warm: a warm-up step (no ranking)."""
    U = res.risk.size
    rec = np.ones(U, bool) if rec is None else rec
    bad = set()
    g = res.gnmr / alpha
    bad |= set(np.flatnonzero(rec & np.isfinite(g) & (np.abs(g - 1.0) <= GUARD)).tolist())
    if window_full:
        d = res.dgnmr / beta
        bad |= set(np.flatnonzero(rec & np.isfinite(d) & (np.abs(d - 1.0) <= GUARD)).tolist())
    if warm:
        return sorted(bad)
    cand = rec & ((res.risk > 1.0) | (lock_before > 0))
    if active_before is not None:
        cand &= ~active_before
    idx = np.flatnonzero(cand)
    if 0 < max_o < idx.size:
        order = idx[np.lexsort((idx, -res.risk[idx]))]
        r_in, r_out = res.risk[order[max_o - 1]], res.risk[order[max_o]]
        if r_in != r_out:
            if (r_in - r_out) <= GUARD * r_in:
                bad.add(int(order[max_o]))
        else:
            r = res.risk[idx]
            above, below = r[r > r_in], r[r < r_in]
            if above.size and above.min() - r_in <= GUARD * above.min():
                bad.add(int(idx[np.flatnonzero(r == above.min())[-1]]))
            if below.size and r_in - below.max() <= GUARD * r_in:
                bad.add(int(idx[np.flatnonzero(r == below.max())[0]]))
    return sorted(bad)


def nudge_factor(j: int) -> float:
    k = (j + 1) // 2
    return 1.0 + (3e-4 * k if j % 2 == 1 else -3e-4 * k)


def guarded_stream(w, norms_of_step, max_nudges: int = 40, budget_mode: int = BUDGET_ACTIVE,
                   warmup_steps: int = 0):
    """Run the oracle over a workload's stream, nudging unit-steps that break
    the guards.  norms_of_step(t, scale32, units) -> {b: norm}.  Returns
    (nudge [T, U] float64, norms [T, U], results, alphas, betas)."""
    if budget_mode not in (BUDGET_ACTIVE, BUDGET_ADMITTED):
        raise ValueError("guards are defined for the active-set and admitted-only budgets")
    T, U = w.steps, w.num_units
    ctl = Controller(U, window=w.window, max_o=w.max_o, lock_len=w.lock_len, eps=w.eps,
                     budget_mode=budget_mode, warmup_steps=warmup_steps)
    nudge = np.ones((T, U))
    norms = np.zeros((T, U))
    results, alphas, betas = [], [], []
    for t in range(1, T + 1):
        alpha, beta = w.alpha(t), w.beta(t)
        scale32 = w.scale32(t, nudge[t - 1])
        nd = norms_of_step(t, scale32, None)
        n = np.array([nd[b] for b in range(U)])
        tries = np.zeros(U, dtype=np.int64)
        while True:
            snap = ctl.get_state()
            res = ctl.step(n, alpha, beta)
            bad = violations(res, alpha, beta, w.max_o, len(snap["Q"]) == w.window,
                             snap["lock"],
                             active_before=(snap["active"] if budget_mode == BUDGET_ADMITTED
                                            else None),
                             warm=t <= warmup_steps)
            if not bad:
                break
            ctl.set_state(snap)
            for b in bad:
                tries[b] += 1
                if tries[b] > max_nudges:
                    raise RuntimeError(f"cannot clear guards for unit {b} at step {t}")
                nudge[t - 1, b] = nudge_factor(int(tries[b]))
            scale32 = w.scale32(t, nudge[t - 1])
            nd = norms_of_step(t, scale32, bad)
            for b in bad:
                n[b] = nd[b]
        norms[t - 1] = n
        results.append(res)
        alphas.append(alpha)
        betas.append(beta)
    return nudge, norms, results, alphas, betas
