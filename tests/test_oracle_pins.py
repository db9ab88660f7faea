"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these re-types the oracle's own formula: each one checks it against
an exact rational computation of the paper's closed-form definitions, a
closed form derived by hand, an invariant stated by the paper, or brute-force
enumeration.  All CPU only.
"""
from fractions import Fraction
from itertools import combinations

import numpy as np
import pytest

from oracle import BF16, F32, Controller, sumsq, unit_norm
from synth import values as V


def rel(a, b):
    a, b = float(a), float(b)
    if a == b:
        return 0.0
    return abs(a - b) / max(abs(a), abs(b))


# --------------------------------------------------------------------------
# norm (Sec. 2, local-gradient equation)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [F32, BF16])
def test_sumsq_matches_exact_rational(dtype):
    x = V.unit_values(seed=3, t=5, b=7, scale=3.7e-3, dtype=dtype, start=11, count=5003)
    y = V.unit_values(seed=3, t=5, b=8, scale=9.1e-5, dtype=dtype, start=0, count=777)
    floats = []
    for arr in (x, y):
        f = V.bf16_bits_to_f32(arr) if dtype == BF16 else arr
        floats.extend(float(v) for v in f)
    exact = sum((Fraction(v) * Fraction(v) for v in floats), Fraction(0))
    got = sumsq([(x, dtype), (y, dtype)])
    assert rel(got, exact) < 1e-13


def test_norm_of_constant_magnitude_is_closed_form():
    # +-c with c = 2^-10 and N = 4096: ||g|| = c * sqrt(N) = 2^-4 exactly.
    signs = np.where(np.arange(4096) % 3 == 0, -1.0, 1.0).astype(np.float32)
    g32 = signs * np.float32(2.0 ** -10)
    assert unit_norm([(g32, F32)]) == 2.0 ** -4
    g16 = V.f32_to_bf16_bits(g32)
    assert unit_norm([(g16, BF16)]) == 2.0 ** -4
    # split into three segments of one unit: the norm of the concatenation
    assert unit_norm([(g16[:100], BF16), (g16[100:101], BF16), (g16[101:], BF16)]) == 2.0 ** -4


def test_norm_empty_unit_is_zero():
    assert unit_norm([]) == 0.0
    assert unit_norm([(np.zeros(0, np.float32), F32)]) == 0.0


def bf16_const(value, n):
    return V.f32_to_bf16_bits(np.full(n, value, dtype=np.float32))


def test_norm_range_ends_at_sum_of_squares_two_to_128():
    # Reading for non-finite norms: the gradient pass accumulates in fp32, so
    # a unit whose sum of squares reaches 2^128 has norm +inf.  Exact cases:
    # two elements of 2^63 sum to 2^127 (norm 2^63.5), four to exactly 2^128.
    assert unit_norm([(bf16_const(2.0 ** 63, 2), BF16)]) == 2.0 ** 63.5
    assert unit_norm([(bf16_const(-(2.0 ** 63), 3), BF16)]) == np.sqrt(3.0) * 2.0 ** 63
    assert unit_norm([(bf16_const(2.0 ** 63, 4), BF16)]) == np.inf
    # one element of 2^64 (its square is 2^128), in a segment of small values
    seg = bf16_const(2.0 ** -10, 1000)
    seg[500] = bf16_const(-(2.0 ** 64), 1)[0]
    assert unit_norm([(seg, BF16)]) == np.inf
    # the largest bf16 below 2^64, alone: finite, exactly its magnitude
    below = (2.0 - 2.0 ** -7) * 2.0 ** 63
    assert unit_norm([(bf16_const(below, 1), BF16)]) == below
    # split over segments, the limit applies to the unit's total
    assert unit_norm([(bf16_const(2.0 ** 63, 2), BF16),
                      (np.full(2, 2.0 ** 63, np.float32), F32)]) == np.inf
    # fp32 values far beyond bf16's grid near the limit: 2^64 * (1 - 2^-24)
    # squared is below 2^128; the sum of two such squares is not
    v = np.float32(2.0 ** 64 * (1 - 2.0 ** -24))
    assert unit_norm([(np.array([v], np.float32), F32)]) == float(v)
    assert unit_norm([(np.array([v, v], np.float32), F32)]) == np.inf


def test_norm_of_non_finite_elements():
    # An Inf element gives an infinite sum of squares, a NaN element a NaN one
    # (NaN wins over Inf), whatever the other elements are.
    seg = bf16_const(2.0 ** -10, 64)
    inf_seg = seg.copy()
    inf_seg[3] = V.f32_to_bf16_bits(np.array([-np.inf], np.float32))[0]
    assert unit_norm([(inf_seg, BF16)]) == np.inf
    nan32 = np.full(9, 0.5, np.float32)
    nan32[8] = np.nan
    assert np.isnan(unit_norm([(nan32, F32)]))
    assert np.isnan(unit_norm([(inf_seg, BF16), (nan32, F32)]))


# --------------------------------------------------------------------------
# GNMR and Delta-GNMR against the closed-form definitions (Sec. 3.1, 3.2)
# --------------------------------------------------------------------------

def exact_gnmr_history(norms):
    """GNMR_t = n_t / ((1/(t-1)) sum_{tau<t} n_tau), GNMR_1 = 1 -- exact."""
    out = []
    for t in range(1, len(norms) + 1):
        if t == 1:
            out.append(Fraction(1))
        else:
            mean = sum((Fraction(v) for v in norms[: t - 1]), Fraction(0)) / (t - 1)
            out.append(Fraction(norms[t - 1]) / mean)
    return out


def exact_dgnmr(gh, t, delta):
    """Delta-GNMR_t = GNMR_t / ((1/delta) sum_{tau=1..delta} GNMR_{t-tau}); 1 while
    fewer than delta previous values exist."""
    if t - 1 < delta:
        return Fraction(1)
    window = gh[t - 1 - delta: t - 1]
    return gh[t - 1] / (sum(window, Fraction(0)) / delta)


@pytest.mark.parametrize("delta", [1, 3, 5])
def test_gnmr_and_dgnmr_follow_definitions(delta):
    rng = np.random.default_rng(11)
    T, U = 40, 3
    norms = np.exp(rng.normal(size=(T, U)))
    ctl = Controller(U, window=delta, max_o=U, lock_len=2, eps=0.0)
    res = [ctl.step(norms[i], 1.3, 1.2) for i in range(T)]
    for b in range(U):
        gh = exact_gnmr_history([norms[i, b] for i in range(T)])
        for t in range(1, T + 1):
            assert rel(res[t - 1].gnmr[b], gh[t - 1]) < 1e-13
            assert rel(res[t - 1].dgnmr[b], exact_dgnmr(gh, t, delta)) < 1e-13


def test_running_mean_is_arithmetic_mean():
    rng = np.random.default_rng(12)
    T = 200
    norms = np.abs(rng.normal(size=(T, 1))) * 1e-3
    ctl = Controller(1, window=5, max_o=1, lock_len=1, eps=0.0)
    for t in range(1, T + 1):
        ctl.step(norms[t - 1], 1.1, 1.5)
        mean = sum((Fraction(v) for v in norms[:t, 0]), Fraction(0)) / t
        assert rel(ctl.A[0], mean) < t * 2e-16


def test_constant_magnitude_gives_exact_ones():
    # constant-magnitude gradients: GNMR = Delta-GNMR = 1 exactly, every step
    rng = np.random.default_rng(0)
    grads = [np.where(rng.random(1000) < 0.5, -c, c).astype(np.float32)
             for c in (2.0 ** -10, 3.3e-4, 7.77e-3)]
    U = len(grads)
    ctl = Controller(U, window=5, max_o=2, lock_len=3, eps=0.0)
    for t in range(1, 31):
        # fresh signs every step, same magnitudes
        norms = [unit_norm([(rng.permutation(g), F32)]) for g in grads]
        r = ctl.step(norms, 1.1, 1.5)
        assert np.all(r.gnmr == 1.0) and np.all(r.dgnmr == 1.0)
        assert np.all(r.risk == max(1 / 1.1, 1 / 1.5))
        assert r.mask.sum() == 0


@pytest.mark.parametrize("k", [10, 20, 50])
@pytest.mark.parametrize("t0", [7, 12])
def test_spike_closed_form(k, t0):
    # constant n for t < t0, k*n at t0, n afterwards (t0 > delta):
    #   GNMR_t0 = k, Delta_t0 = k, A_t0 = n (t0 - 1 + k) / t0,
    #   GNMR_{t0+j} = (t0+j-1) / (t0+j-2+k)                    (j >= 1),
    #   Delta_{t0+1} = delta t0 / ((t0-1+k)(delta-1+k)).
    delta, c, N = 5, 2.0 ** -10, 1024
    g = np.full(N, c, dtype=np.float32)
    g[::2] *= -1
    n = unit_norm([(g, F32)])
    spike = unit_norm([(g * np.float32(k), F32)])
    assert spike == k * n                       # exact: k c is representable
    ctl = Controller(1, window=delta, max_o=1, lock_len=1, eps=0.0)
    T = t0 + 8
    res = []
    for t in range(1, T + 1):
        res.append(ctl.step([spike if t == t0 else n], 1.1, 1.5))
        if t == t0:
            assert rel(ctl.A[0], Fraction(n) * (t0 - 1 + k) / t0) < 1e-15
    r0 = res[t0 - 1]
    assert rel(r0.gnmr[0], k) < 1e-15 and rel(r0.dgnmr[0], k) < 1e-15
    hist = [Fraction(1)] * (t0 - 1) + [Fraction(k)]
    for j in range(1, T - t0 + 1):
        gj = Fraction(t0 + j - 1, t0 + j - 2 + k)
        assert rel(res[t0 + j - 1].gnmr[0], gj) < 1e-14
        window = hist[-delta:]
        dj = gj / (sum(window, Fraction(0)) / delta)
        assert rel(res[t0 + j - 1].dgnmr[0], dj) < 1e-14
        hist.append(gj)
    assert rel(res[t0].dgnmr[0], Fraction(delta * t0, (t0 - 1 + k) * (delta - 1 + k))) < 1e-14
    # the spike itself is selected (R = max(k/1.1, k/1.5) > 1)
    assert r0.mask[0] == 1


def test_scale_invariance_power_of_two():
    # GNMR is dimensionless: scaling a unit's norms by 2^m at every step
    # leaves every ratio, the mask and the locks bitwise unchanged (eps = 0).
    rng = np.random.default_rng(5)
    T, U = 60, 6
    norms = np.exp(rng.normal(scale=0.4, size=(T, U)))
    norms[20, 2] *= 9.0
    norms[33, 4] *= 5.0
    scaled = norms * (2.0 ** np.array([-7, 3, 0, 11, -20, 1]))[None, :]
    a = Controller(U, window=5, max_o=2, lock_len=3, eps=0.0)
    b = Controller(U, window=5, max_o=2, lock_len=3, eps=0.0)
    for t in range(T):
        ra, rb = a.step(norms[t], 1.1, 1.3), b.step(scaled[t], 1.1, 1.3)
        for f in ("gnmr", "dgnmr", "risk", "mask", "lock"):
            assert np.array_equal(getattr(ra, f), getattr(rb, f)), (t, f)


def test_first_steps_are_clamped_to_one():
    ctl = Controller(4, window=3, max_o=4, lock_len=1, eps=1e-12)
    rng = np.random.default_rng(1)
    for t in range(1, 5):
        r = ctl.step(np.abs(rng.normal(size=4)), 1.5, 1.5)
        if t == 1:
            assert np.all(r.gnmr == 1.0)
        if t <= 3:       # fewer than delta previous GNMR values
            assert np.all(r.dgnmr == 1.0)
        else:
            assert not np.all(r.dgnmr == 1.0)


def test_zero_mean_rules():
    # A = 0 (a unit whose every norm so far was 0) gives GNMR = 1; with eps = 0
    # a window of zero GNMRs gives Delta-GNMR = 1 instead of a division by 0.
    ctl = Controller(2, window=2, max_o=2, lock_len=1, eps=0.0)
    seq = [[0.0, 1.0], [0.0, 1.0], [2.0, 0.0], [1.0, 0.0], [1.0, 0.0], [1.0, 3.0]]
    out = [ctl.step(s, 1.1, 1.5) for s in seq]
    assert out[0].gnmr[0] == 1 and out[1].gnmr[0] == 1 and out[2].gnmr[0] == 1
    assert out[3].gnmr[0] == 1.0 / (2.0 / 3.0)     # A after three steps = 2/3
    assert out[3].gnmr[1] == 0.0 and out[4].gnmr[1] == 0.0
    # unit 1 at t=6: window {0, 0} -> Delta = 1 ; GNMR = 3 / (2/5)
    assert out[5].gnmr[1] == 3.0 / (2.0 / 5.0) and out[5].dgnmr[1] == 1.0


# --------------------------------------------------------------------------
# selection and locks (Alg. 2; Cor. 1; Sec. 3.4)
# --------------------------------------------------------------------------

def brute_force_active(R, cand, max_o):
    """Cor. 1: the budgeted set maximises sum R over subsets of the pool of
    size min(maxO, |C|); among maximisers take the lexicographically smallest
    sorted index tuple.  Exact rational sums."""
    C = [b for b in range(len(R)) if cand[b]]
    k = min(max_o, len(C))
    best, best_set = None, None
    for sub in combinations(C, k):
        s = sum((Fraction(float(R[b])) for b in sub), Fraction(0))
        if best is None or s > best or (s == best and sub < best_set):
            best, best_set = s, sub
    return set(best_set or ())


@pytest.mark.parametrize("seed", range(6))
def test_selection_equals_brute_force_and_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    U = int(rng.integers(3, 11))
    max_o = int(rng.integers(0, 5))
    lock_len = int(rng.integers(0, 4))
    rec = rng.random(U) < 0.8
    T = 40
    norms = np.exp(rng.normal(scale=0.6, size=(T, U)))
    # a few exact ties: two units share a norm stream
    if U >= 4:
        norms[:, 3] = norms[:, 1]
    ctl = Controller(U, window=3, max_o=max_o, lock_len=lock_len, eps=0.0, recoverable=rec)
    lock_before = np.zeros(U, dtype=np.int64)
    for t in range(1, T + 1):
        alpha = float(rng.choice([0.6, 1.0, 1.2]))
        beta = float(rng.choice([0.8, 1.1, 1.4]))
        r = ctl.step(norms[t - 1], alpha, beta)
        trig = rec & (r.risk > 1.0)
        cand = trig | (rec & (lock_before > 0))
        A = set(np.flatnonzero(r.mask).tolist())
        assert A == brute_force_active(r.risk, cand, max_o)
        assert len(A) <= max_o                                   # hard cap
        assert all(cand[b] for b in A)                           # A within C
        if trig.sum() >= max_o:                                  # triggered first
            assert all(trig[b] for b in A)
        if cand.sum() <= max_o:                                  # cap, not quota
            assert A == set(np.flatnonzero(cand).tolist())
        assert np.all((r.lock >= 0) & (r.lock <= lock_len))
        assert all(r.mask[b] for b in np.flatnonzero(r.lock > 0))
        assert np.all(r.lock[~rec] == 0)
        assert r.stats["n_active"] == len(A) and r.stats["n_cand"] == cand.sum()
        lock_before = r.lock.astype(np.int64)


@pytest.mark.parametrize("lock_len", [0, 1, 4, 8])
def test_lock_holds_exactly_lock_len_steps(lock_len):
    # one spike at t0, no competition: unit 0 is active for steps
    # t0 .. t0 + T_lock and inactive from t0 + T_lock + 1 on.
    U, t0 = 3, 9
    T = t0 + lock_len + 5
    ctl = Controller(U, window=5, max_o=2, lock_len=lock_len, eps=0.0)
    active_steps = []
    for t in range(1, T + 1):
        n = np.ones(U)
        if t == t0:
            n[0] = 4.0
        r = ctl.step(n, 1.5, 1.5)
        if r.mask[0]:
            active_steps.append(t)
        assert r.mask[1:].sum() == 0
    assert active_steps == list(range(t0, t0 + lock_len + 1))


def test_eviction_clears_lock():
    # unit 0 locked; then maxO = 1 others trigger harder -> unit 0 evicted, lock 0
    ctl = Controller(3, window=5, max_o=1, lock_len=5, eps=0.0)
    for t in range(1, 9):
        ctl.step([1.0, 1.0, 1.0], 1.5, 1.5)
    r = ctl.step([3.0, 1.0, 1.0], 1.5, 1.5)
    assert r.mask.tolist() == [1, 0, 0] and r.lock[0] == 5
    r = ctl.step([1.0, 9.0, 1.0], 1.5, 1.5)
    assert r.mask.tolist() == [0, 1, 0] and r.lock.tolist() == [0, 5, 0]
    r = ctl.step([1.0, 1.0, 1.0], 1.5, 1.5)
    assert r.mask.tolist() == [0, 1, 0] and r.lock.tolist() == [0, 4, 0]


def test_retrigger_while_locked_resets_lock():
    ctl = Controller(2, window=5, max_o=2, lock_len=3, eps=0.0)
    for t in range(1, 8):
        ctl.step([1.0, 1.0], 1.5, 1.5)
    assert ctl.step([4.0, 1.0], 1.5, 1.5).lock[0] == 3
    assert ctl.step([1.0, 1.0], 1.5, 1.5).lock[0] == 2
    assert ctl.step([9.0, 1.0], 1.5, 1.5).lock[0] == 3


def test_zero_budget_selects_nothing():
    rng = np.random.default_rng(2)
    ctl = Controller(5, window=2, max_o=0, lock_len=3, eps=1e-12)
    for t in range(20):
        r = ctl.step(np.exp(rng.normal(size=5)) * (10 if t == 10 else 1), 0.4, 0.5)
        assert r.mask.sum() == 0 and r.lock.sum() == 0
        assert r.stats["hit_maxo"] == 1


def test_alpha_below_one_is_pure_top_k():
    # alpha = 0.4 (the paper's 4-bit stress setting): every unit triggers, the
    # active set is the maxO largest R every step.
    rng = np.random.default_rng(3)
    U, max_o = 12, 4
    ctl = Controller(U, window=5, max_o=max_o, lock_len=1, eps=1e-12)
    for t in range(30):
        r = ctl.step(np.exp(rng.normal(scale=0.2, size=U)), 0.4, 1.5)
        assert r.stats["n_trig"] == U and r.stats["n_active"] == max_o
        top = np.lexsort((np.arange(U), -r.risk))[:max_o]
        assert set(np.flatnonzero(r.mask)) == set(top.tolist())


def test_non_recoverable_units_are_monitored_only():
    ctl = Controller(3, window=5, max_o=3, lock_len=2, eps=0.0, recoverable=[1, 0, 1])
    for t in range(1, 8):
        ctl.step([1.0, 1.0, 1.0], 1.5, 1.5)
    r = ctl.step([5.0, 5.0, 1.0], 1.5, 1.5)
    assert r.risk[1] > 1 and r.mask.tolist() == [1, 0, 0] and r.lock[1] == 0


def test_snapshot_restore_is_bitwise():
    rng = np.random.default_rng(4)
    U = 9
    norms = np.exp(rng.normal(size=(30, U)))
    ctl = Controller(U, window=5, max_o=3, lock_len=4, eps=1e-12)
    for t in range(12):
        ctl.step(norms[t], 1.1, 1.3)
    snap = ctl.get_state()
    first = [ctl.step(norms[t], 1.1, 1.3) for t in range(12, 30)]
    ctl2 = Controller(U, window=5, max_o=3, lock_len=4, eps=1e-12)
    ctl2.set_state(snap)
    second = [ctl2.step(norms[t], 1.1, 1.3) for t in range(12, 30)]
    for a, b in zip(first, second):
        for f in ("gnmr", "dgnmr", "risk", "mask", "lock"):
            assert np.array_equal(getattr(a, f), getattr(b, f))


def test_non_finite_norm_is_flagged_and_ranked_first():
    ctl = Controller(3, window=2, max_o=1, lock_len=2, eps=1e-12)
    for t in range(4):
        ctl.step([1.0, 2.0, 3.0], 1.1, 1.5)
    A_before = ctl.A.copy()
    r = ctl.step([np.nan, 50.0, np.inf], 1.1, 1.5)
    assert r.stats["n_nonfinite"] == 2
    assert np.isinf(r.risk[0]) and np.isinf(r.risk[2])
    assert r.mask.tolist() == [1, 0, 0]           # +inf ties -> smaller index
    assert ctl.A[0] == A_before[0] and ctl.A[2] == A_before[2]
    assert ctl.Q[-1][0] == 1.0


def test_invalid_arguments_raise():
    with pytest.raises(ValueError):
        Controller(0, 5, 1, 1, 0.0)
    with pytest.raises(ValueError):
        Controller(3, 0, 1, 1, 0.0)
    with pytest.raises(ValueError):
        Controller(3, 5, -1, 1, 0.0)
    ctl = Controller(3, 5, 1, 1, 0.0)
    with pytest.raises(ValueError):
        ctl.step([1, 1, 1], 0.0, 1.5)
    with pytest.raises(ValueError):
        ctl.step([1, 1, 1], 1.1, float("nan"))


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_native_sumsq_matches_exact_rational_and_numpy(dtype):
    from oracle import native

    x = V.unit_values(seed=4, t=2, b=1, scale=2.3e-3, dtype=dtype, start=3, count=4001)
    f = V.bf16_bits_to_f32(x) if dtype == BF16 else x
    exact = sum((Fraction(float(v)) ** 2 for v in f), Fraction(0))
    got = native.sumsq(x, dtype)
    assert rel(got, exact) < 4001 * 1.2e-16
    big = V.unit_values(seed=4, t=2, b=2, scale=2.3e-3, dtype=dtype, start=0, count=3_000_001)
    assert rel(native.sumsq(big, dtype), sumsq([(big, dtype)])) < 1e-10


def test_eps_enters_both_denominators():
    # GNMR_t = n_t / (A_{t-1} + eps), Delta_t = GNMR_t / (mean(Q) + eps) (Alg. 1),
    # checked with a large eps in exact rationals.
    eps, delta = 0.5, 2
    norms = [1.0, 3.0, 2.0, 4.0, 1.5]
    ctl = Controller(1, window=delta, max_o=1, lock_len=1, eps=eps)
    A, Q = Fraction(0), []
    for t, n in enumerate(norms, start=1):
        r = ctl.step([n], 1.1, 1.5)
        G = Fraction(1) if (t == 1 or A == 0) else Fraction(n) / (A + Fraction(eps))
        D = G / (sum(Q, Fraction(0)) / delta + Fraction(eps)) if len(Q) == delta else Fraction(1)
        assert rel(r.gnmr[0], G) < 1e-15 and rel(r.dgnmr[0], D) < 1e-15
        A = A + (Fraction(n) - A) / t
        Q = (Q + [G])[-delta:]


def test_trigger_is_strict():
    # constant magnitude with alpha = 1: R = GNMR / alpha = 1 exactly, which is
    # not a trigger (Alg. 2 uses R > 1)
    ctl = Controller(2, window=3, max_o=2, lock_len=2, eps=0.0)
    for t in range(10):
        r = ctl.step([0.25, 4.0], 1.0, 1.0)
        assert np.all(r.risk == 1.0) and r.mask.sum() == 0 and r.stats["n_trig"] == 0


# --------------------------------------------------------------------------
# policy variants: admitted-only budget (App. C remark), warm-up (App. E.6)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_admitted_only_budget_brute_force(seed):
    from oracle import BUDGET_ADMITTED

    rng = np.random.default_rng(200 + seed)
    U, max_o, lock_len, T = 9, 2, 3, 40
    norms = np.exp(rng.normal(scale=0.5, size=(T, U)))
    ctl = Controller(U, window=3, max_o=max_o, lock_len=lock_len, eps=0.0,
                     budget_mode=BUDGET_ADMITTED)
    prev_active = np.zeros(U, bool)
    lock_before = np.zeros(U, np.int64)
    grew = False
    for t in range(1, T + 1):
        r = ctl.step(norms[t - 1], 1.05, 1.1)
        cand = (r.risk > 1.0) | (lock_before > 0)
        A = r.mask.astype(bool)
        keep = cand & prev_active
        assert np.array_equal(A & prev_active, keep)           # continuing units retained
        assert not np.any(A & ~cand)                            # A_t within C_t
        new = A & ~prev_active
        assert new.sum() <= max_o                               # cap on admissions only
        pool = cand & ~prev_active
        assert set(np.flatnonzero(new)) == brute_force_active(r.risk, pool, max_o)
        grew |= A.sum() > max_o
        prev_active, lock_before = A, r.lock.astype(np.int64)
    assert grew                    # the active set itself may exceed maxO in this mode


def test_admitted_only_equals_active_cap_when_nothing_was_active():
    from oracle import BUDGET_ADMITTED

    rng = np.random.default_rng(9)
    U = 30
    norms = np.exp(rng.normal(scale=0.5, size=(2, U)))
    # alpha = 0.05: every unit triggers at t = 1 and 2; lock 0.  At t = 1
    # (A_0 empty) the two conventions agree; at t = 2 the admitted-only budget
    # keeps the 4 active units and admits 4 more.
    a = Controller(U, 5, 4, 0, 0.0)
    b = Controller(U, 5, 4, 0, 0.0, budget_mode=BUDGET_ADMITTED)
    ra, rb = a.step(norms[0], 0.05, 1.5), b.step(norms[0], 0.05, 1.5)
    assert ra.mask.sum() == 4 and np.array_equal(ra.mask, rb.mask)
    first = rb.mask.astype(bool)
    ra, rb = a.step(norms[1], 0.05, 1.5), b.step(norms[1], 0.05, 1.5)
    assert ra.stats["n_trig"] == U and rb.stats["n_trig"] == U
    assert ra.mask.sum() == 4 and rb.mask.sum() == 8
    assert np.all(rb.mask[first] == 1)

@pytest.mark.parametrize("max_o", [0, 3])
def test_warmup_all_recover_then_normal(max_o):
    rng = np.random.default_rng(21)
    U, T, W = 12, 30, 5
    rec = np.ones(U, bool)
    rec[[2, 7]] = False
    norms = np.exp(rng.normal(scale=0.3, size=(T, U)))
    norms[W - 1, 4] *= 8.0                      # a trigger in the last warm-up step
    warm = Controller(U, 5, max_o, 4, 1e-12, recoverable=rec, warmup_steps=W)
    plain = Controller(U, 5, max_o, 4, 1e-12, recoverable=rec)
    for t in range(1, T + 1):
        rw, rp = warm.step(norms[t - 1], 1.3, 1.5), plain.step(norms[t - 1], 1.3, 1.5)
        for f in ("norm", "gnmr", "dgnmr", "risk"):               # statistics untouched
            assert np.array_equal(getattr(rw, f), getattr(rp, f))
        if t <= W:
            assert np.array_equal(rw.mask.astype(bool), rec)        # everyone recovers
            assert rw.stats["n_active"] == rec.sum() and rw.stats["hit_maxo"] == 0
        else:
            assert rw.mask.sum() <= max_o
    # the lock of the warm-up trigger carries over: Alg. 2's rule on A_W = B_rec
    w2 = Controller(U, 5, max_o, 4, 1e-12, recoverable=rec, warmup_steps=W)
    for t in range(1, W + 1):
        r = w2.step(norms[t - 1], 1.3, 1.5)
    assert r.lock[4] == 4 and r.risk[4] > 1.0


@pytest.mark.parametrize("W,K", [(1, 3), (6, 4), (10, 0)])
def test_static_baseline_top_k_by_mean_gnmr(W, K):
    # App. E.4: all units recover during the W profiling steps; then the K
    # recoverable units with the largest mean GNMR over steps 1..W are the
    # fixed recovery set (ties to the smaller index); no locks.
    from oracle import BUDGET_STATIC

    rng = np.random.default_rng(40 + W)
    U, T = 10, W + 6
    rec = np.ones(U, bool)
    rec[3] = False
    norms = np.exp(rng.normal(scale=0.4, size=(T, U)))
    ctl = Controller(U, 5, K, 4, 0.0, recoverable=rec, budget_mode=BUDGET_STATIC, warmup_steps=W)
    res = [ctl.step(norms[t], 1.1, 1.5) for t in range(T)]
    means = []
    for b in range(U):
        gh = exact_gnmr_history([norms[i, b] for i in range(W)])
        means.append(sum(gh, Fraction(0)) / W)
    want = sorted((b for b in range(U) if rec[b]), key=lambda b: (-means[b], b))[:K]
    for t, r in enumerate(res, start=1):
        assert np.all(r.lock == 0)
        if t <= W:
            assert np.array_equal(r.mask.astype(bool), rec)
        else:
            assert set(np.flatnonzero(r.mask)) == set(want), t
    assert res[W].stats["hit_maxo"] == int(rec.sum() > 0 and rec.sum() >= K)
    with pytest.raises(ValueError):
        Controller(U, 5, K, 4, 0.0, budget_mode=BUDGET_STATIC, warmup_steps=0)
