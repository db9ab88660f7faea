"""Pins of the quantisation-simulated linear operator's oracle (App. E.2)
against an independent route: exact rational products written out element
by element, correctly rounded to bf16 by enumerating neighbouring bf16
values, and each row quantised on its own by the (separately pinned)
per-token quantiser.  Planted mistakes in a copy of the oracle must each fail
one of these pins.  CPU only."""
import importlib.util
import os
import sys
from fractions import Fraction

import numpy as np
import pytest

from oracle import fakequant as FQ
from oracle import qsim as QS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def bf16_value(bits):
    return Fraction(float(FQ.bf16_to_f32(np.array([bits], np.uint16))[0]))


def nearest_bf16(v: Fraction) -> int:
    """The bf16 bit pattern nearest to the rational v (ties to the even
    pattern), found among the neighbours of its float32 truncation."""
    f = np.float32(float(v))
    base = int(np.array([f], np.float32).view(np.uint32)[0] >> 16)
    cands = set()
    for b in range(base - 2, base + 3):
        for s in (0, 0x8000):
            p = (b & 0x7FFF) | s
            if (p & 0x7F80) != 0x7F80:            # finite patterns only
                cands.add(p)
    best = min(cands, key=lambda p: (abs(bf16_value(p) - v), p & 1, p))
    if bf16_value(best) == 0:
        return 0x8000 if v < 0 else 0
    return best


def brute_matmul(a_bits, b_bits):
    """bf16(a b) element by element with exact rationals."""
    r, k = a_bits.shape
    c = b_bits.shape[1]
    out = np.zeros((r, c), np.uint16)
    for i in range(r):
        for j in range(c):
            s = sum((bf16_value(a_bits[i, t]) * bf16_value(b_bits[t, j]) for t in range(k)),
                    Fraction(0))
            out[i, j] = nearest_bf16(s)
    return out


def rows_each(bits, fmt):
    """Every row quantised on its own (one row at a time)."""
    return np.stack([FQ.fakequant_rows(bits[i:i + 1], fmt)[0] for i in range(bits.shape[0])])


def operands(seed, T=5, d_in=8, d_out=16, spread=True):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(T, d_in)) * (10.0 ** rng.uniform(-2, 1, (T, 1)))
    w = rng.normal(size=(d_out, d_in)) * (10.0 ** rng.uniform(-3, 0, (d_out, 1)))
    if spread:
        w[1] *= 2.0 ** -20                       # one output channel far smaller
    dy = rng.normal(size=(T, d_out)) * (10.0 ** rng.uniform(-3, 0, (T, 1)))
    return (FQ.f32_to_bf16(x.astype(np.float32)), FQ.f32_to_bf16(w.astype(np.float32)),
            FQ.f32_to_bf16(dy.astype(np.float32)))


@pytest.mark.parametrize("fmt", [0, 1, 2, 3, 4, 5])
def test_each_quantisation_point_by_brute_force(fmt):
    x, w, dy = operands(fmt)
    f = QS.forward(x, w, fmt)
    x_q, w_q = rows_each(x, fmt), rows_each(w, fmt)
    assert np.array_equal(f["x_q"], x_q)
    assert np.array_equal(f["w_q"], w_q)                 # one scale per output channel
    y = brute_matmul(x_q, w_q.T)
    assert np.array_equal(f["y"], y)
    assert np.array_equal(f["y_q"], rows_each(y, fmt))
    b = QS.backward(dy, f["x_q"], f["w_q"], fmt)
    dy_q = rows_each(dy, fmt)
    assert np.array_equal(b["dy_q"], dy_q)
    dx = brute_matmul(dy_q, w_q)
    assert np.array_equal(b["dx"], dx)
    assert np.array_equal(b["dx_q"], rows_each(dx, fmt))
    dw = brute_matmul(dy_q.T, x_q)
    assert np.array_equal(b["dw"], dw)
    assert np.array_equal(b["dw_q"], rows_each(dw, fmt))


def test_identity_format_is_the_plain_bf16_layer():
    x, w, dy = operands(9)
    f = QS.forward(x, w, 0)
    b = QS.backward(dy, f["x_q"], f["w_q"], 0)
    assert np.array_equal(f["y_q"], brute_matmul(x, w.T))
    assert np.array_equal(b["dx_q"], brute_matmul(dy, w))
    assert np.array_equal(b["dw_q"], brute_matmul(dy.T, x))


def test_on_grid_operands_pass_through_unchanged():
    # rows on the E2M1 grid whose largest magnitude is the format's maximum
    # (scale 1) are fixed points of the quantiser: the operator then computes
    # with the operands themselves
    rng = np.random.default_rng(4)
    g = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], np.float32)
    def on_grid(r, c):
        v = rng.choice(g, size=(r, c)) * rng.choice([-1, 1], size=(r, c))
        v[:, 0] = 6.0
        return FQ.f32_to_bf16(v.astype(np.float32))
    x, w = on_grid(4, 8), on_grid(8, 8)
    f = QS.forward(x, w, 1)
    assert np.array_equal(f["x_q"], x) and np.array_equal(f["w_q"], w)
    assert np.array_equal(f["y"], brute_matmul(x, w.T))


def test_small_output_channel_keeps_its_own_scale():
    x, w, dy = operands(2)
    f = QS.forward(x, w, 1)
    wf, qf = FQ.bf16_to_f32(w), FQ.bf16_to_f32(f["w_q"])
    # the 2^-20 channel is quantised on its own scale: not flushed to zero, and
    # within the E2M1 grid's relative error of its row maximum
    assert np.any(qf[1] != 0)
    assert np.all(np.abs(qf[1] - wf[1]) <= np.abs(wf[1]).max() / 6 * 0.5 * (1 + 2 ** -7))


def test_formats_follow_the_controller_decision():
    low, rec = (1, 1), (3, 4)
    assert QS.formats(False, low, rec) == low
    assert QS.formats(True, low, rec) == rec


# -- pin strength --------------------------------------------------------------

SRC = os.path.join(ROOT, "oracle", "qsim.py")
MUTANTS = [
    ("weights quantised per input column", "w_q = fakequant_rows(w_bits, fmt)",
     "w_q = fakequant_rows(w_bits.T, fmt).T"),
    ("forward with the unquantised input", "y = matmul_bf16(x_q, w_q.T)",
     "y = matmul_bf16(x_bits, w_q.T)"),
    ("output not quantised", '"y_q": fakequant_rows(y, fmt)', '"y_q": y'),
    ("dx from the unquantised dy", "dx = matmul_bf16(dy_q, w_q)", "dx = matmul_bf16(dy_bits, w_q)"),
    ("dw from the unquantised dy", "dw = matmul_bf16(dy_q.T, x_q)",
     "dw = matmul_bf16(dy_bits.T, x_q)"),
    ("dx not quantised", '"dx_q": fakequant_rows(dx, fmt)', '"dx_q": dx'),
    ("dw not quantised", '"dw_q": fakequant_rows(dw, fmt)', '"dw_q": dw'),
    ("dw quantised per column", '"dw_q": fakequant_rows(dw, fmt)',
     '"dw_q": fakequant_rows(dw.T, fmt).T'),
    ("formats swapped", "return recovery if in_recovery else low",
     "return low if in_recovery else recovery"),
]
PINS = [(test_each_quantisation_point_by_brute_force, dict(fmt=1)),
        (test_each_quantisation_point_by_brute_force, dict(fmt=4)),
        (test_identity_format_is_the_plain_bf16_layer, {}),
        (test_on_grid_operands_pass_through_unchanged, {}),
        (test_small_output_channel_keeps_its_own_scale, {}),
        (test_formats_follow_the_controller_decision, {})]


def mutant(original, planted):
    src = open(SRC).read()
    assert original in src, original
    spec = importlib.util.spec_from_loader("oracle.qsim_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"                   # its relative imports resolve in oracle/
    sys.modules["oracle.qsim_mutant"] = mod
    try:
        exec(compile(src.replace(original, planted, 1), "qsim_mutant", "exec"), mod.__dict__)
    finally:
        del sys.modules["oracle.qsim_mutant"]
    return mod


@pytest.mark.parametrize("name,original,planted", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, original, planted):
    global QS
    real = QS
    caught = []
    try:
        QS = mutant(original, planted)
        for fn, kw in PINS:
            try:
                fn(**kw)
            except (AssertionError, ValueError, IndexError):
                caught.append(fn.__name__)
    finally:
        QS = real
    assert caught, f"no pin fails for the planted mistake: {name}"


def test_unmutated_oracle_passes_every_listed_pin():
    for fn, kw in PINS:
        fn(**kw)
