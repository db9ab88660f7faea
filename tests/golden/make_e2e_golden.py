"""Writes tests/golden/e2e_<workload>.npz: the oracle's expected controller
outputs for every step of a full-size synthetic workload.

Inputs come from the seeded generator (synth: the recipe, and the C host twin
of the counter-based values).  Norms come from the oracle's plain-C float64
sum of squares (oracle/native.py), and every step runs the oracle controller
(oracle/gnmr_oracle.py) with the guard co-simulation of tests/streams.py,
which nudges a unit-step's scale when a decision would sit within 1e-4 of
its threshold.  Nothing here touches the HIP library.

Stored per workload:
  nudge_t, nudge_b, nudge_f  the nudged unit-steps (1-based step, unit, factor)
  mask_bits    np.packbits of the [T, U] active-set masks (axis 1)
  lock         uint8 [T, U] lock counters after each step
  stats        int64 [T, 8] counters (t, n_trig_gnmr, n_trig_dgnmr, n_trig,
               n_cand, n_active, hit_maxo, n_nonfinite)
  norm32       float32 [len(norm_steps), U] oracle norms (float32 is far inside
               the 1e-5 bar) at the 1-based steps norm_steps: every step, or for
               workloads of more than 400k unit-steps steps 1, 2 and every 16th
  sample       int64 [S] unit indices with float64 gnmr/dgnmr/risk [T, S]
  gnmr_all, dgnmr_all  float32 [len(norm_steps), U] GNMR and Delta-GNMR of every
               unit at the norm steps (workloads of more than 300 units, whose
               sample above is a subset)
  rot_period, rot_norm32, rot_gnmr32, rot_dgnmr32, rot_risk32  (workloads of
               more than 300 units) the norm, GNMR, Delta-GNMR and R of a
               rotating set of units at every step: at step t the units
               u = (t - 1) % P, (t - 1) % P + P, ... with P = rot_period, laid end
               to end in step order, so that every step checks about U / P units
               and every unit is checked at about T / P steps

Policy variants (App. C budget remark, App. E.6 warm-up) are written under
their own names (VARIANTS below) from the same stream, with the controller
run under that policy; their files also hold budget_mode and warmup_steps.

Usage: python tests/golden/make_e2e_golden.py [workload ...] [--threads N]
       python tests/golden/make_e2e_golden.py --thin workload ...   (rewrite an
       existing file with the norm subsampling above)
"""
from __future__ import annotations

import argparse
import math
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

import streams as S  # noqa: E402
from oracle import native  # noqa: E402
from synth import host  # noqa: E402
from synth import recipe as R  # noqa: E402

from oracle import BUDGET_ACTIVE, BUDGET_ADMITTED  # noqa: E402

# name -> (workload, budget_mode, warm-up steps): the admitted-only budget with
# the high-fidelity warm-up over the first 5% of the steps (App. E.6), on the
# MoE stream, whose pools of about 1,500 candidates make maxO = 32 bind.
VARIANTS = {
    "moe-admitted-warmup": ("moe", BUDGET_ADMITTED, math.ceil(0.05 * R.get("moe").steps)),
}

CHUNK = 1 << 22
FULL_NORMS_MAX = 400_000      # unit-steps up to which every step's norms are kept
ROT_UNITS = 700               # units per step of the rotating set (about)
STAT_KEYS = ("t", "n_trig_gnmr", "n_trig_dgnmr", "n_trig", "n_cand", "n_active", "hit_maxo",
             "n_nonfinite")


def golden_path(name: str) -> str:
    return os.path.join(HERE, f"e2e_{name}.npz")


def norm_steps_for(steps: int, units: int) -> np.ndarray:
    if steps * units <= FULL_NORMS_MAX:
        return np.arange(1, steps + 1, dtype=np.int64)
    return np.array([t for t in range(1, steps + 1) if t <= 2 or t % 16 == 0], dtype=np.int64)


def rot_period(units: int) -> int:
    return -(-units // ROT_UNITS)


def rot_units(t: int, units: int) -> np.ndarray:
    """The rotating set of units whose outputs are stored at 1-based step t."""
    p = rot_period(units)
    return np.arange((t - 1) % p, units, p, dtype=np.int64)


def thin(name: str) -> str:
    """Rewrite a golden file keeping norms only at norm_steps_for(...)."""
    path = golden_path(name)
    z = np.load(path, allow_pickle=False)
    d = {k: z[k] for k in z.files}
    T, U = int(d["steps"]), int(d["units"])
    keep = norm_steps_for(T, U)
    old = d.get("norm_steps", np.arange(1, T + 1, dtype=np.int64))
    rows = [int(np.flatnonzero(old == t)[0]) for t in keep]
    d["norm32"] = d["norm32"][rows]
    d["norm_steps"] = keep
    np.savez_compressed(path, **d)
    return path


def unit_norm(seed, t, b, scale32, dtype, numel):
    buf = np.empty(min(CHUNK, max(numel, 1)), dtype=np.float32 if dtype == 0 else np.uint16)
    s = 0.0
    for lo in range(0, numel, CHUNK):
        n = min(CHUNK, numel - lo)
        host.unit_values(seed, t, b, scale32, dtype, lo, n, out=buf[:n])
        s += native.sumsq(buf[:n], dtype)
    return math.sqrt(s)


def make(name: str, threads: int) -> str:
    base, budget_mode, warmup = VARIANTS.get(name, (name, BUDGET_ACTIVE, 0))
    w = R.get(base)
    U, T = w.num_units, w.steps
    pool = ThreadPoolExecutor(max_workers=threads)
    t_start = time.time()

    def norms_of_step(t, scale32, units):
        sel = range(U) if units is None else units
        vals = pool.map(lambda b: unit_norm(w.seed, t, b, float(scale32[b]), w.units[b].dtype,
                                            w.units[b].numel), sel)
        out = dict(zip(sel, vals))
        if units is None:
            print(f"  {name} t={t}/{T} ({time.time() - t_start:.0f} s)", flush=True)
        return out

    nudge, norms, res, _, _ = S.guarded_stream(w, norms_of_step, budget_mode=budget_mode,
                                               warmup_steps=warmup)
    pool.shutdown()
    masks = np.stack([r.mask for r in res]).astype(np.uint8)
    locks = np.stack([r.lock for r in res])
    assert locks.max() <= 255
    stats = np.array([[r.stats[k] for k in STAT_KEYS] for r in res], dtype=np.int64)
    rng = np.random.default_rng(7)
    ever = np.flatnonzero(masks.any(axis=0))
    sample = np.unique(np.concatenate([
        np.arange(U) if U <= 300 else rng.choice(U, 192, replace=False),
        ever[:64], [0, U - 1]])).astype(np.int64)
    nt, nb = np.nonzero(nudge != 1.0)
    out = golden_path(name)
    np.savez_compressed(
        out, workload=base, budget_mode=budget_mode, warmup_steps=warmup, steps=T, units=U,
        nudge_t=(nt + 1).astype(np.int64), nudge_b=nb.astype(np.int64),
        nudge_f=nudge[nt, nb],
        mask_bits=np.packbits(masks, axis=1), lock=locks.astype(np.uint8), stats=stats,
        norm_steps=norm_steps_for(T, U),
        norm32=norms[norm_steps_for(T, U) - 1].astype(np.float32), sample=sample,
        gnmr=np.stack([r.gnmr[sample] for r in res]),
        dgnmr=np.stack([r.dgnmr[sample] for r in res]),
        risk=np.stack([r.risk[sample] for r in res]),
        **({} if U <= 300 else {
            "gnmr_all": np.stack([res[t - 1].gnmr for t in norm_steps_for(T, U)]).astype(
                np.float32),
            "dgnmr_all": np.stack([res[t - 1].dgnmr for t in norm_steps_for(T, U)]).astype(
                np.float32),
            "rot_period": np.int64(rot_period(U)),
            "rot_norm32": np.concatenate([norms[t - 1][rot_units(t, U)]
                                          for t in range(1, T + 1)]).astype(np.float32),
            **{f"rot_{f}32": np.concatenate([getattr(res[t - 1], f)[rot_units(t, U)]
                                             for t in range(1, T + 1)]).astype(np.float32)
               for f in ("gnmr", "dgnmr", "risk")}}))
    print(f"{name}: {T} steps x {U} units, {len(nt)} nudged unit-steps, "
          f"{int(masks.sum())} active unit-steps, {time.time() - t_start:.0f} s -> {out}",
          flush=True)
    return out


def load(name: str) -> dict:
    z = np.load(golden_path(name), allow_pickle=False)
    d = {k: z[k] for k in z.files}
    d["mask"] = np.unpackbits(d["mask_bits"], axis=1, count=int(d["units"])).astype(np.uint8)
    if "norm_steps" not in d:
        d["norm_steps"] = np.arange(1, int(d["steps"]) + 1, dtype=np.int64)
    d.setdefault("budget_mode", np.int64(BUDGET_ACTIVE))
    d.setdefault("warmup_steps", np.int64(0))
    return d


def nudge_table(d: dict) -> np.ndarray:
    nudge = np.ones((int(d["steps"]), int(d["units"])))
    nudge[d["nudge_t"] - 1, d["nudge_b"]] = d["nudge_f"]
    return nudge


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("workloads", nargs="*",
                    default=["tiny", "llama2-7b", "llama2-13b", "moe", "fine128", "fine32"])
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 8)
    ap.add_argument("--thin", action="store_true")
    a = ap.parse_args()
    for n in a.workloads:
        print(thin(n) if a.thin else make(n, a.threads), flush=True)
