"""Strength of the oracle pins: plausible mistakes are planted into a copy of
the oracle (on the CPU, never in the real one) and at least one pin must fail
for each.  CPU only."""
import importlib.util
import os
import sys
import types

import pytest

import test_fakequant_oracle as FP
import test_oracle_pins as P

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")
SRC = os.path.join(ORACLE, "gnmr_oracle.py")

# (name, original text, planted mistake)
MUTANTS = [
    ("running mean over t+1", "A_next = self.A + (n - self.A) / t",
     "A_next = self.A + (n - self.A) / (t + 1)"),
    ("window mean over delta+1", "den = total / delta + eps", "den = total / (delta + 1) + eps"),
    ("eps subtracted", "n[has_mean] / (self.A[has_mean] + eps)",
     "n[has_mean] / (self.A[has_mean] - eps)"),
    ("eps dropped from window", "den = total / delta + eps", "den = total / delta"),
    ("queue keeps delta+1", "if len(self.Q) > delta:", "if len(self.Q) > delta + 1:"),
    ("min instead of max", "risk = np.maximum(g_term, d_term)", "risk = np.minimum(g_term, d_term)"),
    ("alpha and beta swapped", "g_term = gnmr / alpha", "g_term = gnmr / beta"),
    ("non-strict trigger", "triggered = self.rec & (risk > 1.0)",
     "triggered = self.rec & (risk >= 1.0)"),
    ("locks ignored in pool", "cand = triggered | (self.rec & (self.lock > 0))",
     "cand = triggered"),
    ("non-recoverable selectable", "triggered = self.rec & (risk > 1.0)",
     "triggered = (risk > 1.0)"),
    ("ascending selection", "order = np.lexsort((pool_idx, -risk[pool_idx]))",
     "order = np.lexsort((pool_idx, risk[pool_idx]))"),
    ("ties to larger index", "order = np.lexsort((pool_idx, -risk[pool_idx]))",
     "order = np.lexsort((-pool_idx, -risk[pool_idx]))"),
    ("lock set to T_lock - 1", "new_lock[b] = self.lock_len", "new_lock[b] = self.lock_len - 1"),
    ("lock not decremented", "new_lock[b] = max(self.lock[b] - 1, 0)",
     "new_lock[b] = max(self.lock[b], 0)"),
    ("eviction keeps lock", "new_lock = np.zeros(U, dtype=np.int64)", "new_lock = self.lock.copy()"),
    ("budget off by one", "if pool_idx.size <= self.max_o:", "if pool_idx.size <= self.max_o + 1:"),
    ("L1 instead of L2", "s += float(np.dot(x, x))", "s += float(np.sum(np.abs(x)))"),
    ("bf16 widened wrongly", "<< np.uint32(16)", "<< np.uint32(15)"),
    ("GNMR not clamped at A = 0", "has_mean = finite & (self.A != 0.0)", "has_mean = finite"),
    ("admitted mode keeps every candidate", "keep = cand & self.active", "keep = cand"),
    ("warm-up ignored", "cand = self.rec.copy()", "cand = cand"),
    ("static set ranked ascending", "order = np.lexsort((ranked, -mean[ranked]))",
     "order = np.lexsort((ranked, mean[ranked]))"),
    ("static mean over W+1 steps", "mean = self.gsum / W", "mean = self.gsum / (W + 1) - self.gsum * 0 + (np.arange(U) == 0)"),
    ("current GNMR in window", "for q in self.Q:                       # oldest to newest",
     "for q in self.Q[1:] + [gnmr]:"),
    ("no sum-of-squares range limit", "if ss >= SUMSQ_LIMIT:", "if ss > SUMSQ_LIMIT * 4:"),
    ("range limit on the norm, not its square", "if ss >= SUMSQ_LIMIT:",
     "if ss >= 2.0 ** 64:"),
    ("range limit strict", "if ss >= SUMSQ_LIMIT:", "if ss > SUMSQ_LIMIT:"),
]

PINS = [
    (P.test_sumsq_matches_exact_rational, dict(dtype=P.BF16)),
    (P.test_norm_of_constant_magnitude_is_closed_form, {}),
    (P.test_norm_range_ends_at_sum_of_squares_two_to_128, {}),
    (P.test_norm_of_non_finite_elements, {}),
    (P.test_gnmr_and_dgnmr_follow_definitions, dict(delta=3)),
    (P.test_running_mean_is_arithmetic_mean, {}),
    (P.test_constant_magnitude_gives_exact_ones, {}),
    (P.test_spike_closed_form, dict(k=20, t0=7)),
    (P.test_zero_mean_rules, {}),
    (P.test_selection_equals_brute_force_and_invariants, dict(seed=0)),
    (P.test_selection_equals_brute_force_and_invariants, dict(seed=3)),
    (P.test_lock_holds_exactly_lock_len_steps, dict(lock_len=4)),
    (P.test_eviction_clears_lock, {}),
    (P.test_alpha_below_one_is_pure_top_k, {}),
    (P.test_non_recoverable_units_are_monitored_only, {}),
    (P.test_eps_enters_both_denominators, {}),
    (P.test_trigger_is_strict, {}),
    (P.test_admitted_only_budget_brute_force, dict(seed=0)),
    (P.test_warmup_all_recover_then_normal, dict(max_o=3)),
    (P.test_static_baseline_top_k_by_mean_gnmr, dict(W=6, K=4)),
]


def mutant_module(original: str, planted: str, path: str = SRC) -> types.ModuleType:
    src = open(path).read()
    assert original in src, f"mutation anchor not found: {original!r}"
    spec = importlib.util.spec_from_loader("oracle_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    sys.modules["oracle_mutant"] = mod          # dataclasses look the module up
    try:
        exec(compile(src.replace(original, planted, 1), "oracle_mutant", "exec"), mod.__dict__)
    finally:
        del sys.modules["oracle_mutant"]
    return mod


@pytest.mark.parametrize("name,original,planted", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, original, planted):
    mod = mutant_module(original, planted)
    for attr in ("Controller", "sumsq", "unit_norm"):
        monkeypatch.setattr(P, attr, getattr(mod, attr))
    caught = []
    for fn, kw in PINS:
        try:
            fn(**kw)
        except (AssertionError, ValueError, IndexError, ZeroDivisionError, FloatingPointError):
            caught.append(fn.__name__)
    assert caught, f"no pin fails for the planted mistake: {name}"


def test_unmutated_oracle_passes_every_listed_pin():
    for fn, kw in PINS:
        fn(**kw)


# The actuator oracle (per-token fake quantisation) and its pins.
FQ_MUTANTS = [
    ("float ties away from zero", "q = np.rint(a / step) * step",
     "q = np.floor(a / step + 0.5) * step"),
    ("float no saturation", "q = np.minimum(q, fmax)", "q = q"),
    ("E4M3 max 480", "3: (3, -6, 448.0)", "3: (3, -6, 480.0)"),
    ("E2M1 subnormal binade off by one", "1: (1, 0, 6.0)", "1: (1, -1, 6.0)"),
    ("E5M2 as E5M3", "4: (2, -14, 57344.0)", "4: (3, -14, 57344.0)"),
    ("float sign dropped", "return np.copysign(q, y).astype(np.float32)     #",
     "return q.astype(np.float32)     #"),
    ("int ties away from zero", "q = np.minimum(np.rint(np.abs(y).astype(np.float64)), qmax)",
     "q = np.minimum(np.floor(np.abs(y).astype(np.float64) + 0.5), qmax)"),
    ("int clamp at 128", "q = np.minimum(np.rint(np.abs(y).astype(np.float64)), qmax)",
     "q = np.minimum(np.rint(np.abs(y).astype(np.float64)), qmax + 1)"),
    ("int grid to 128", "INT_FORMATS = {5: 127.0}", "INT_FORMATS = {5: 128.0}"),
    ("int truncates", "q = np.minimum(np.rint(np.abs(y).astype(np.float64)), qmax)",
     "q = np.minimum(np.trunc(np.abs(y).astype(np.float64)), qmax)"),
    ("zero token keeps -0", "out = np.where(nz, out, np.float32(0.0))", "out = out"),
    ("scale from the column maximum", "amax = np.max(np.abs(x), axis=1, keepdims=True)",
     "amax = np.max(np.abs(x), axis=0, keepdims=True)"),
    ("bf16 rounds half away", "r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1)))",
     "r = (u + np.uint64(0x8000))"),
    ("bf16 truncates", "r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1)))",
     "r = u"),
    ("low and recovery formats swapped", "fmt_hi if m else fmt_lo", "fmt_lo if m else fmt_hi"),
]

FQ_PINS = [fn for name, fn in sorted(vars(FP).items())
           if name.startswith("test_") and callable(fn)]


def run_fq_pin(fn):
    names = fn.__code__.co_varnames[:fn.__code__.co_argcount]
    if names == ("fmt",):
        for fmt in (1, 2, 3, 4):
            fn(fmt)
    else:
        fn()


@pytest.mark.parametrize("name,original,planted", FQ_MUTANTS, ids=[m[0] for m in FQ_MUTANTS])
def test_actuator_pins_catch_planted_mistake(monkeypatch, name, original, planted):
    mod = mutant_module(original, planted, os.path.join(ORACLE, "fakequant.py"))
    monkeypatch.setattr(FP, "FQ", mod)
    caught = []
    for fn in FQ_PINS:
        try:
            run_fq_pin(fn)
        except (AssertionError, ValueError, IndexError, KeyError, ZeroDivisionError):
            caught.append(fn.__name__)
    assert caught, f"no pin fails for the planted mistake: {name}"


def test_unmutated_actuator_oracle_passes_every_pin():
    assert len(FQ_PINS) >= 6
    for fn in FQ_PINS:
        run_fq_pin(fn)
