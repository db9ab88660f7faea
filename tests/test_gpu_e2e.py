"""End-to-end parity on every step of every workload, at full size.

The expected outputs (tests/golden/e2e_<workload>.npz) were written by
tests/golden/make_e2e_golden.py from the oracle alone: host-generated
gradients, the oracle's float64 norms and controller, and guard nudges that
keep every decision at least 1e-4 from its threshold.  Here the same
gradients are generated on the device (the HIP generator is bit-identical to
the host twin) and run through gnmr_step in the benchmark's launch
configuration (the policy-variant files under the policy they were written
with).  Masks, locks and counters must match bit for bit at every
step; norms, GNMR, Delta-GNMR and R of every unit at the stored steps (every
step, or steps 1, 2 and every 16th on the longest streams), of a stored
sample of units at every step, and (workloads of more than 300 units) of a
rotating set of about 700 units at every step that visits every unit, within
1e-5.
"""
import sys

import numpy as np
import pytest

from golden.make_e2e_golden import golden_path, load, nudge_table, rot_units
from gpu_util import controller_for, device_buffer, require_gpu
from synth import layout as L
from synth import recipe as R

pytestmark = pytest.mark.gpu

E2E = ["tiny", "llama2-7b", "llama2-13b", "llama2-13b-layers", "moe", "fine128", "fine32",
       "moe-admitted-warmup"]
STAT_KEYS = ("t", "n_trig_gnmr", "n_trig_dgnmr", "n_trig", "n_cand", "n_active", "hit_maxo",
             "n_nonfinite")


@pytest.fixture(scope="module")
def gen():
    require_gpu()
    from synth.gpu import Generator

    return Generator()


@pytest.mark.parametrize("name", E2E)
def test_e2e_every_step_matches_oracle(gen, name):
    torch = require_gpu()
    d = load(name)
    w = R.get(str(d["workload"]))
    policy = dict(budget_mode=int(d["budget_mode"]), warmup_steps=int(d["warmup_steps"]))
    assert int(d["units"]) == w.num_units and int(d["steps"]) == w.steps
    nudge = nudge_table(d)
    sample = d["sample"]
    lay = L.for_workload(w)
    print(f"e2e {name}: {w.steps} steps x {w.num_units} units, {policy}, "
          f"{len(d['nudge_t'])} nudged unit-steps ({golden_path(name)})", flush=True)
    sys.stdout.flush()
    buf, base, ptrs = device_buffer(torch, lay)
    active = 0
    rot_at = 0  # offset of this step's rotating set in the rot_* arrays
    try:
        with controller_for(lay, w, ptrs, **policy) as ctl:
            for t in range(1, w.steps + 1):
                gen.fill(lay, base, w.seed, t, w.scale32(t, nudge[t - 1]))
                ctl.step(w.alpha(t), w.beta(t))
                out = ctl.query()
                what = f"{name} t={t}"
                bad = np.flatnonzero(out["mask"] != d["mask"][t - 1])
                assert bad.size == 0, f"{what}: mask differs at units {bad[:10]}"
                bad = np.flatnonzero(out["lock"] != d["lock"][t - 1])
                assert bad.size == 0, f"{what}: lock differs at units {bad[:10]}"
                got = [out["stats"][k] for k in STAT_KEYS]
                assert got == d["stats"][t - 1].tolist(), f"{what}: stats {got}"
                rows = np.flatnonzero(d["norm_steps"] == t)
                if rows.size:
                    np.testing.assert_allclose(out["norm"], d["norm32"][rows[0]], rtol=1e-5,
                                               atol=0, err_msg=f"{what} norm")
                if rows.size and "gnmr_all" in d:
                    # every unit's ratios at the stored steps; R = max(G/alpha, D/beta)
                    g, dd = d["gnmr_all"][rows[0]], d["dgnmr_all"][rows[0]]
                    np.testing.assert_allclose(out["gnmr"], g, rtol=1e-5, atol=0,
                                               err_msg=f"{what} gnmr (all units)")
                    np.testing.assert_allclose(out["dgnmr"], dd, rtol=1e-5, atol=0,
                                               err_msg=f"{what} dgnmr (all units)")
                    r = np.maximum(g.astype(np.float64) / w.alpha(t),
                                   dd.astype(np.float64) / w.beta(t))
                    np.testing.assert_allclose(out["risk"], r, rtol=1e-5, atol=0,
                                               err_msg=f"{what} risk (all units)")
                for f in ("gnmr", "dgnmr", "risk"):
                    np.testing.assert_allclose(out[f][sample], d[f][t - 1], rtol=1e-5, atol=0,
                                               err_msg=f"{what} {f}")
                if "rot_period" in d:
                    # the rotating set of units stored for this step
                    ru = rot_units(t, w.num_units)
                    sl = slice(rot_at, rot_at + ru.size)
                    rot_at += ru.size
                    for f, key in (("norm", "rot_norm32"), ("gnmr", "rot_gnmr32"),
                                   ("dgnmr", "rot_dgnmr32"), ("risk", "rot_risk32")):
                        np.testing.assert_allclose(out[f][ru], d[key][sl], rtol=1e-5, atol=0,
                                                   err_msg=f"{what} {f} (rotating set)")
                active += int(out["mask"].sum())
        print(f"  {name}: all {w.steps} steps match, {active} active unit-steps", flush=True)
    finally:
        del buf
        torch.cuda.empty_cache()
