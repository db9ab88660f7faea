"""The stored end-to-end expectations (tests/golden/e2e_*.npz) are consistent
with themselves: the rotating per-step sets agree with the all-unit arrays
at the steps where both exist, R is max(GNMR / alpha_t, Delta-GNMR / beta_t)
of the stored ratios, masks respect the budget, and the counters agree with
the masks.  CPU only; nothing here runs the oracle or the library."""
import numpy as np
import pytest

from golden.make_e2e_golden import load, rot_units
from synth import recipe as R

NAMES = ["tiny", "llama2-7b", "llama2-13b", "llama2-13b-layers", "moe", "fine128", "fine32",
         "moe-admitted-warmup"]
BUDGET_ACTIVE = 0


@pytest.mark.parametrize("name", NAMES)
def test_golden_is_self_consistent(name):
    d = load(name)
    w = R.get(str(d["workload"]))
    T, U = int(d["steps"]), int(d["units"])
    assert (T, U) == (w.steps, w.num_units)
    mask, lock, stats = d["mask"], d["lock"], d["stats"]
    assert mask.shape == (T, U) and lock.shape == (T, U) and stats.shape == (T, 8)
    assert np.array_equal(stats[:, 0], np.arange(1, T + 1))          # t
    assert np.array_equal(stats[:, 5], mask.sum(axis=1))             # n_active
    if int(d["budget_mode"]) == BUDGET_ACTIVE:
        assert (mask.sum(axis=1) <= w.max_o).all()                   # |A_t| <= maxO
    assert (lock <= w.lock_len).all() and ((lock > 0) <= (mask > 0)).all()
    # the sampled ratios give the sampled risks
    s = d["sample"]
    for t in range(1, T + 1):
        r = np.maximum(d["gnmr"][t - 1] / w.alpha(t), d["dgnmr"][t - 1] / w.beta(t))
        np.testing.assert_allclose(d["risk"][t - 1], r, rtol=1e-15, atol=0)
    if "rot_period" not in d:
        assert U <= 300
        return
    # the rotating sets tile the steps in order and visit every unit
    sizes = [rot_units(t, U).size for t in range(1, T + 1)]
    assert d["rot_norm32"].size == sum(sizes)
    seen = np.zeros(U, bool)
    at = 0
    for t in range(1, T + 1):
        ru = rot_units(t, U)
        sl = slice(at, at + ru.size)
        at += ru.size
        seen[ru] = True
        g, dd = d["rot_gnmr32"][sl], d["rot_dgnmr32"][sl]
        r = np.maximum(g.astype(np.float64) / w.alpha(t), dd.astype(np.float64) / w.beta(t))
        np.testing.assert_allclose(d["rot_risk32"][sl], r, rtol=1e-6, atol=0)
        row = np.flatnonzero(d["norm_steps"] == t)
        if row.size:          # where the all-unit arrays exist, they hold the same values
            assert np.array_equal(d["rot_norm32"][sl], d["norm32"][row[0]][ru])
            assert np.array_equal(g, d["gnmr_all"][row[0]][ru])
            assert np.array_equal(dd, d["dgnmr_all"][row[0]][ru])
        common, i_s, i_r = np.intersect1d(s, ru, return_indices=True)
        np.testing.assert_allclose(g[i_r], d["gnmr"][t - 1][i_s], rtol=1e-7, atol=0)
    assert seen.all() or T < int(d["rot_period"])
