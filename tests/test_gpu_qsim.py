"""The quantisation-simulated linear operator of App. E.2 (QuantSimLinears:
K4 quantisations around library GEMMs) against its oracle (oracle/qsim.py).

Bars:
  * x_q, w_q and dy_q (quantisations of inputs): bit-exact;
  * on data whose products sum exactly in fp32 (operands on a format grid
    with their rows' maximum at the format's largest value): every tensor,
    y, y_q, dx, dx_q, dw and dw_q included, bit-exact;
  * on random data: the products within the fp32-accumulation bound of the
    exact product (oracle/wgrad.py), and the quantised products within one
    grid step of the oracle's, plus that bound (a product that lands near a
    rounding boundary of the format may round the other way);
  * the formats follow the controller's mask; a short training loop with the
    controller stepping over the quantised weight gradients matches the
    oracle controller step for step.
"""
import numpy as np
import pytest

from gpu_util import assert_step_matches, require_gpu
from oracle import fakequant as FQ
from oracle import qsim as QS
from oracle import wgrad as W

pytestmark = pytest.mark.gpu

BF16, E2M1, E3M2, E4M3, E5M2 = 0, 1, 2, 3, 4


def bits(t):
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(
        -1, t.shape[-1])


def from_bits(torch, b):
    return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).to("cuda").view(
        torch.bfloat16)


def grid_rows(rng, rows, cols, fmt):
    """Rows whose largest magnitude is the format's largest value (scale 1)
    and whose other values are off the grid at 1/64 of it."""
    amax = FQ.fmax_of(fmt)
    x = rng.integers(-63, 64, size=(rows, cols)).astype(np.float32) * np.float32(amax / 64)
    x[np.arange(rows), rng.integers(0, cols, rows)] = np.where(rng.random(rows) < 0.5, amax,
                                                               -amax)
    return FQ.f32_to_bf16(x)


def step_of(q_bits, fmt):
    """Per element, the grid step of the format at the element's magnitude,
    in the row's scale (row maximum / fmax); bf16 bits in."""
    if fmt == BF16:
        return np.zeros(q_bits.shape)
    mbits, emin, fmax = FQ.FORMATS[fmt] if fmt in FQ.FORMATS else (None, None, 127.0)
    v = np.abs(FQ.bf16_to_f32(q_bits).astype(np.float64))
    s = v.max(axis=1, keepdims=True) / fmax
    s = np.where(s > 0, s, 1.0)
    if mbits is None:                                   # INT8: unit steps
        return np.broadcast_to(s, v.shape)
    _, E = np.frexp(np.maximum(v / s, 2.0 ** emin))
    return np.exp2(np.maximum(E - 1.0, emin) - mbits) * s


def assert_quantised_near(got, want, exact_bound, fmt, what):
    """Quantised products: within one grid step (at the larger magnitude) of
    the oracle's, plus twice the product's error bound (the oracle's product
    is the exact one rounded to bf16, the device's within the bound of the
    exact one) and two bf16 roundings of the rescaled values."""
    g = FQ.bf16_to_f32(got).astype(np.float64)
    w = FQ.bf16_to_f32(want).astype(np.float64)
    step = np.maximum(step_of(got, fmt), step_of(want, fmt))
    tol = step * (1 + 2.0 ** -6) + 2 * exact_bound + 2.0 ** -7 * np.abs(w) + 2.0 ** -126
    bad = np.abs(g - w) > tol
    assert not bad.any(), (what, np.argwhere(bad)[:5], g[bad][:5], w[bad][:5])
    return float(np.mean(got == want))


def run_layer(torch, x_bits, w_bits, dy_bits, low, rec, in_recovery):
    """One forward and backward of a one-layer controller setup whose mask
    puts the unit in A_t or not; returns the captured tensors."""
    from paper_2606_00539_amd.torch_units import QuantSimLinears, TorchUnits

    out_f, in_f = w_bits.shape
    lin = torch.nn.Linear(in_f, out_f, bias=False).to("cuda", torch.bfloat16)
    with torch.no_grad():
        lin.weight.copy_(from_bits(torch, w_bits).view(out_f, in_f))
    units = TorchUnits([("lin.weight", lin.weight)], max_o=1, lock_len=0, eps=1e-12,
                       unit_of=lambda n: "lin")
    op = QuantSimLinears(units, [("lin", lin)], low=low, recovery=rec, capture=True)
    try:
        if in_recovery:
            # a first step: with alpha < 1 every unit is a candidate, so the one unit
            # enters A_t (the gradient it reads is any valid bf16 tensor)
            lin.weight.grad = torch.zeros_like(lin.weight)
            units.step(0.4, 1.5)
            assert units.query()["mask"].tolist() == [1]
            lin.weight.grad = None
        x = from_bits(torch, x_bits).view(x_bits.shape).requires_grad_(True)
        y = lin(x)
        y.backward(from_bits(torch, dy_bits).view(dy_bits.shape))
        torch.cuda.synchronize()
        cap = {k: bits(v) for k, v in op.captured["lin"].items() if v is not None}
        cap["weight_grad"] = bits(lin.weight.grad)
        cap["x_grad"] = bits(x.grad)
        cap["out"] = bits(y)
        return cap
    finally:
        op.close()
        units.close()


@pytest.mark.parametrize("in_recovery", [False, True])
def test_operator_bit_exact_on_exact_data(in_recovery):
    torch = require_gpu()
    rng = np.random.default_rng(40 + in_recovery)
    low, rec = (E2M1, E2M1), (E3M2, E3M2)
    f_fmt, b_fmt = QS.formats(in_recovery, low, rec)
    T, d_in, d_out = 48, 64, 40
    x, w, dy = grid_rows(rng, T, d_in, f_fmt), grid_rows(rng, d_out, d_in, f_fmt), \
        grid_rows(rng, T, d_out, b_fmt)
    cap = run_layer(torch, x, w, dy, low, rec, in_recovery)
    f = QS.forward(x, w, f_fmt)
    b = QS.backward(dy, f["x_q"], f["w_q"], b_fmt)
    want = {**f, **b}
    for k in ("x_q", "w_q", "y", "y_q", "dy_q", "dx_q", "dw_q"):
        assert np.array_equal(cap[k], want[k]), (k, np.argwhere(cap[k] != want[k])[:5])
    assert np.array_equal(cap["out"], want["y_q"])
    assert np.array_equal(cap["weight_grad"], want["dw_q"])
    assert np.array_equal(cap["x_grad"], want["dx_q"])
    assert not np.array_equal(want["x_q"], x)           # the quantisation is visible


@pytest.mark.parametrize("in_recovery", [False, True])
def test_operator_random_data_within_bounds(in_recovery):
    torch = require_gpu()
    rng = np.random.default_rng(50 + in_recovery)
    low, rec = (E2M1, E2M1), (E4M3, E5M2)                # the paper's hybrid FP8 recovery
    f_fmt, b_fmt = QS.formats(in_recovery, low, rec)
    T, d_in, d_out = 96, 200, 136
    x = FQ.f32_to_bf16((rng.normal(size=(T, d_in)) *
                        10.0 ** rng.uniform(-2, 1, (T, 1))).astype(np.float32))
    w = FQ.f32_to_bf16((rng.normal(size=(d_out, d_in)) * 0.05).astype(np.float32))
    dy = FQ.f32_to_bf16((rng.normal(size=(T, d_out)) *
                         10.0 ** rng.uniform(-4, -1, (T, 1))).astype(np.float32))
    cap = run_layer(torch, x, w, dy, low, rec, in_recovery)
    f = QS.forward(x, w, f_fmt)
    b = QS.backward(dy, f["x_q"], f["w_q"], b_fmt)
    for k, want in (("x_q", f["x_q"]), ("w_q", f["w_q"]), ("dy_q", b["dy_q"])):
        assert np.array_equal(cap[k], want), k
    # the products, against the exact product of the (bit-exact) quantised operands
    e_y = W.widen_bf16(f["x_q"]) @ W.widen_bf16(f["w_q"]).T
    b_y = W.error_bound(f["x_q"].T, f["w_q"].T, e_y)
    assert np.all(np.abs(W.widen_bf16(cap["y"]) - e_y) <= b_y)
    e_dx = W.widen_bf16(b["dy_q"]) @ W.widen_bf16(f["w_q"])
    b_dx = W.error_bound(b["dy_q"].T, f["w_q"], e_dx)
    e_dw = W.widen_bf16(b["dy_q"]).T @ W.widen_bf16(f["x_q"])
    b_dw = W.error_bound(b["dy_q"], f["x_q"], e_dw)
    match = [assert_quantised_near(cap["y_q"], f["y_q"], b_y, f_fmt, "y_q"),
             assert_quantised_near(cap["dx_q"], b["dx_q"], b_dx, b_fmt, "dx_q"),
             assert_quantised_near(cap["dw_q"], b["dw_q"], b_dw, b_fmt, "dw_q")]
    assert min(match) > 0.9, match
    assert np.array_equal(cap["weight_grad"], cap["dw_q"])
    assert np.array_equal(cap["x_grad"], cap["dx_q"])


def test_training_loop_with_the_controller_in_the_loop():
    """Eight SGD steps of a two-block SwiGLU stack whose six projections run
    the simulated operator (E2M1 low-cost path, E4M3/E5M2 recovery path), the
    controller stepping over their quantised weight gradients.  Every step:
    the controller matches the oracle fed with the stored gradients' norms
    (masks, locks, counters bit-exact); every layer quantised its input,
    weight and incoming gradient in the formats of the previous step's mask,
    bit for bit; and its weight gradient is the oracle's dw_q within the
    bounds above."""
    torch = require_gpu()
    import torch.nn.functional as F

    from oracle import Controller as Oracle
    from oracle import unit_norm
    from paper_2606_00539_amd.torch_units import QuantSimLinears, TorchUnits, llama_linear_units

    torch.manual_seed(5)
    d, f = 64, 128
    model = torch.nn.ModuleDict({"layers": torch.nn.ModuleList([
        torch.nn.ModuleDict({"gate_proj": torch.nn.Linear(d, f, bias=False),
                             "up_proj": torch.nn.Linear(d, f, bias=False),
                             "down_proj": torch.nn.Linear(f, d, bias=False)})
        for _ in range(2)])}).to("cuda", torch.bfloat16)
    units = TorchUnits(list(model.named_parameters()), max_o=2, lock_len=1, eps=1e-12,
                       unit_of=llama_linear_units)
    U = len(units.unit_names)
    named = [(n, m) for n, m in model.named_modules() if n in units.unit_names]
    low, rec = (E2M1, E2M1), (E4M3, E5M2)
    op = QuantSimLinears(units, named, low=low, recovery=rec, capture=True)
    inputs = {}
    hooks = [m.register_forward_pre_hook(
        lambda mod, args, n=n: inputs.__setitem__(n, bits(args[0]))) for n, m in named]
    ora = Oracle(U, window=5, max_o=2, lock_len=1, eps=1e-12)
    opt = torch.optim.SGD(model.parameters(), lr=0.5)
    mask_prev = np.zeros(U, np.uint8)
    recovered = 0
    try:
        for t in range(1, 9):
            weights = {n: bits(m.weight) for n, m in named}
            x = torch.randn(2, 16, d, device="cuda").to(torch.bfloat16)
            h = x
            for blk in model["layers"]:
                h = h + blk["down_proj"](F.silu(blk["gate_proj"](h)) * blk["up_proj"](h))
            (h.float() ** 2).mean().backward()
            for b, n in enumerate(units.unit_names):
                cap = {k: bits(v) for k, v in op.captured[n].items() if v is not None}
                f_fmt, b_fmt = QS.formats(bool(mask_prev[b]), low, rec)
                fo = QS.forward(inputs[n], weights[n], f_fmt)
                assert np.array_equal(cap["x_q"], fo["x_q"]), (t, n)
                assert np.array_equal(cap["w_q"], fo["w_q"]), (t, n)
                bo = QS.backward(cap["dy"], fo["x_q"], fo["w_q"], b_fmt)
                assert np.array_equal(cap["dy_q"], bo["dy_q"]), (t, n)
                e_dw = W.widen_bf16(bo["dy_q"]).T @ W.widen_bf16(fo["x_q"])
                assert_quantised_near(bits(dict(named)[n].weight.grad), bo["dw_q"],
                                      W.error_bound(bo["dy_q"], fo["x_q"], e_dw), b_fmt,
                                      f"t={t} {n} dw_q")
            units.step(0.9, 1.5)                      # alpha < 1: every unit a candidate
            out = units.query()
            norms = [unit_norm([(bits(p.grad).ravel(), 1)]) for p in units.params]
            ref = ora.step(norms, 0.9, 1.5)
            # this seeded run's decisions are far from their thresholds
            assert np.all(np.abs(ref.gnmr / 0.9 - 1) > 1e-4), t
            assert t <= 5 or np.all(np.abs(ref.dgnmr / 1.5 - 1) > 1e-4), t
            top = np.sort(ref.risk)[::-1]
            # the cut between the 2nd and 3rd largest R: an exact tie (both sides
            # compute it identically, e.g. GNMR = 1 at t = 1) or a clear gap
            assert top[1] == top[2] or top[1] - top[2] > 1e-4 * top[1], t
            assert_step_matches(out, ref, rtol=1e-5, what=f"t={t}")
            recovered += int(out["mask"].sum())
            mask_prev = out["mask"].copy()
            opt.step()
            opt.zero_grad(set_to_none=True)
        assert recovered > 0
    finally:
        for hk in hooks:
            hk.remove()
        op.close()
        units.close()
