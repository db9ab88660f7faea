"""The guard co-simulation's rules (tests/streams.py) on hand-made oracle
results: which unit-steps it flags for a nudge.  CPU only."""
from types import SimpleNamespace

import numpy as np

import streams as S


def result(risk, gnmr=None, dgnmr=None):
    risk = np.asarray(risk, dtype=np.float64)
    ones = np.full(risk.size, 5.0)          # ratios far from both thresholds
    return SimpleNamespace(risk=risk, gnmr=ones if gnmr is None else np.asarray(gnmr),
                           dgnmr=ones if dgnmr is None else np.asarray(dgnmr))


def test_g1_flags_ratios_near_a_threshold():
    r = result([3.0, 3.0, 3.0], gnmr=[1.5 * (1 + 5e-5), 3.0, 3.0], dgnmr=[5, 5, 1.5 * 0.99995])
    assert S.violations(r, 1.5, 1.5, 8, True, np.zeros(3)) == [0, 2]
    # Delta-GNMR is not a decision until the window is full
    assert S.violations(r, 1.5, 1.5, 8, False, np.zeros(3)) == [0]


def test_g2_flags_a_near_tie_at_the_cut():
    # max_o = 2: the 2nd and 3rd largest R of the pool decide the cut
    r = result([4.0, 2.0, 2.0 * (1 - 5e-5), 1.5])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(4)) == [2]
    r = result([4.0, 2.0, 1.9, 1.5])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(4)) == []


def test_g2_exact_tie_needs_clear_neighbours():
    # an exact tie at the cut is computed identically on both sides ...
    r = result([4.0, 2.0, 2.0, 1.5])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(4)) == []
    # ... but a unit just above or just below the tied value could cross it
    r = result([2.0 * (1 + 5e-5), 2.0, 2.0, 1.5])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(4)) == [0]
    r = result([4.0, 2.0, 2.0, 2.0 * (1 - 5e-5)])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(4)) == [3]


def test_g2_ranks_only_new_candidates_under_the_admitted_budget():
    # units 0 and 1 were active: under the admitted-only budget only 2, 3, 4 rank
    r = result([2.0, 2.0 * (1 - 5e-5), 1.9, 1.8, 1.8 * (1 - 5e-5)])
    active = np.array([True, True, False, False, False])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(5), active_before=active) == [4]
    # under the active-set cap all five rank: the cut (maxO = 2) falls between 2.0(1 - 5e-5)
    # and 1.9, far apart; with maxO = 1 it falls inside the near-tie of units 0 and 1
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(5)) == []
    assert S.violations(r, 1.0, 1.0, 1, True, np.zeros(5)) == [1]


def test_no_cut_in_a_warm_up_step():
    r = result([4.0, 2.0, 2.0 * (1 - 5e-5), 1.5])
    assert S.violations(r, 1.0, 1.0, 2, True, np.zeros(4), warm=True) == []


def test_locked_units_join_the_pool():
    # R <= 1 but locked: still a candidate, so it takes part in the cut
    r = result([4.0, 0.9, 0.9 * (1 - 5e-5)])
    lock = np.array([0, 1, 1])
    assert S.violations(r, 1.0, 1.0, 1, True, lock) == []
    assert S.violations(r, 1.0, 1.0, 2, True, lock) == [2]
