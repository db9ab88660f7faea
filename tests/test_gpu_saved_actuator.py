"""The recovery actuator on saved activations only (QuantizedSavedInputs):
the forward product reads the bf16 input, and only the copy kept for the
weight gradient is fake-quantised per token by K4, in the format the unit's
mask entry picks (Sec. 5.1; App. E.2, recoverable scope; App. E.4).

Bars:
  * the forward output is bit-equal to the plain layer's;
  * dW = dy^T x_q with x_q the oracle's per-token quantisation
    (oracle/fakequant.py): bit-exact through K5 on data whose products sum
    exactly, within oracle/wgrad.py's bound through torch's product
    otherwise;
  * dx = dy W, unaffected by the quantisation;
  * the format follows the controller's mask: E2M1 before any step, the
    recovery format for the unit a controller step puts in A_t.
"""
import numpy as np
import pytest

from gpu_util import require_gpu
from oracle import fakequant as FQ
from oracle import wgrad as W

pytestmark = pytest.mark.gpu

E2M1, E3M2 = 1, 2


def bits(t):
    return t.detach().contiguous().view(torch_int16()).cpu().numpy().view(np.uint16).reshape(
        -1, t.shape[-1])


def torch_int16():
    import torch
    return torch.int16


def from_bits(torch, b, shape):
    return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).to("cuda").view(
        torch.bfloat16).reshape(shape)


def grid_rows(rng, rows, cols, amax):
    """bf16 rows with largest magnitude exactly amax and other values off the
    E2M1/E3M2 grids (multiples of amax/64), so that the quantised copy
    differs from the input while its values stay on a coarse grid."""
    x = rng.integers(-63, 64, size=(rows, cols)).astype(np.float32) * np.float32(amax / 64.0)
    x[np.arange(rows), rng.integers(0, cols, rows)] = np.where(rng.random(rows) < 0.5, amax,
                                                               -amax)
    return FQ.f32_to_bf16(x)


def test_fused_saved_quantisation_bit_exact_and_follows_mask():
    torch = require_gpu()
    import torch.nn.functional as F

    from paper_2606_00539_amd.torch_units import FusedWgradUnits, QuantizedSavedInputs

    rng = np.random.default_rng(5)
    T, d_in = 48, 64
    outs = {"a": 40, "b": 48}
    layers = {n: torch.nn.Linear(d_in, o, bias=False).to("cuda", torch.bfloat16)
              for n, o in outs.items()}
    with torch.no_grad():
        for n, m in layers.items():
            w = rng.integers(-3, 4, size=m.weight.shape).astype(np.float32)
            m.weight.copy_(torch.from_numpy(w).to(torch.bfloat16))
    units = FusedWgradUnits(list(layers.items()), max_o=1, lock_len=0, eps=1e-12)
    quant = QuantizedSavedInputs(units, list(layers.items()), E2M1, E3M2)
    try:
        # step 1: no controller step yet, every unit on the low-cost path (E2M1);
        # step 2: after a step with alpha < 1 (every unit a candidate, R tied)
        # maxO = 1 puts unit 0 ("a") in A_t, so "a" saves E3M2, "b" E2M1
        for step, fmts in ((1, {"a": E2M1, "b": E2M1}), (2, {"a": E3M2, "b": E2M1})):
            xs, gs, ys = {}, {}, {}
            for n, m in layers.items():
                amax = 6.0 if fmts[n] == E2M1 else 28.0   # the format's largest value
                xb = grid_rows(rng, T, d_in, amax)
                x = from_bits(torch, xb, (T, d_in)).requires_grad_(True)
                gb = FQ.f32_to_bf16(rng.integers(-4, 5, size=(T, outs[n])).astype(np.float32))
                g = from_bits(torch, gb, (T, outs[n]))
                y = m(x)
                assert torch.equal(y, F.linear(x.detach(), m.weight.detach())), (step, n)
                (y * g).sum().backward()          # dy = g exactly
                xs[n], gs[n], ys[n] = (xb, x), gb, y
            for n, m in layers.items():
                xb, x = xs[n]
                xq = FQ.fakequant_rows(xb, fmts[n])
                assert not np.array_equal(xq, xb)     # the quantisation is visible
                want = W.bf16_rne(W.wgrad_exact(gs[n], xq))
                got = bits(m.weight.grad)
                assert np.array_equal(got, want), (step, n, np.flatnonzero(got != want)[:8])
                # dx = dy W from the unquantised path
                dx = torch.matmul(from_bits(torch, gs[n], (T, outs[n])), m.weight.detach())
                assert torch.equal(x.grad, dx), (step, n)
            units.step(0.4, 1.5)
            if step == 1:
                assert units.query()["mask"].tolist() == [1, 0]
            for m in layers.values():
                m.weight.grad = None
    finally:
        quant.close()
        units.close()


def test_torch_path_saved_quantisation_within_bound():
    """TorchUnits with QuantizedSavedInputs: the weight gradient is torch's
    product dy^T x_q (hipBLASLt), within the fp32-accumulation bound of the
    oracle's exact product; 3-D inputs, a biased layer, random data."""
    torch = require_gpu()
    import torch.nn.functional as F

    from paper_2606_00539_amd.torch_units import QuantizedSavedInputs, TorchUnits

    torch.manual_seed(7)
    d_in = 96
    model = torch.nn.ModuleDict({"a": torch.nn.Linear(d_in, 80, bias=False),
                                 "b": torch.nn.Linear(d_in, 136, bias=True)}).to(
        "cuda", torch.bfloat16)
    units = TorchUnits(model.named_parameters(), max_o=1, lock_len=0, eps=1e-12,
                       unit_of=lambda n: n.split(".")[0] if n.endswith("weight") else None)
    quant = QuantizedSavedInputs(units, list(model.named_children()), E2M1, E3M2)
    try:
        for step, fmts in ((1, {"a": E2M1, "b": E2M1}), (2, {"a": E3M2, "b": E2M1})):
            x = torch.randn(2, 24, d_in, device="cuda").to(torch.bfloat16).requires_grad_(True)
            dys = {}
            ys = {n: model[n](x) for n in ("a", "b")}
            for n, y in ys.items():
                ref = F.linear(x.detach(), model[n].weight.detach(),
                               None if model[n].bias is None else model[n].bias.detach())
                assert torch.equal(y, ref), (step, n)
                y.register_hook(lambda g, n=n: dys.__setitem__(n, g.detach().clone()))
            loss = sum((y.float() ** 2).mean() for y in ys.values())
            loss.backward()
            xb = bits(x)
            dx = sum(torch.matmul(dys[n], model[n].weight.detach()) for n in ("a", "b"))
            torch.testing.assert_close(x.grad.float(), dx.float(), rtol=2e-2, atol=1e-3)
            for n in ("a", "b"):
                xq = FQ.fakequant_rows(xb, fmts[n])
                dyb = bits(dys[n])
                exact = W.wgrad_exact(dyb, xq)
                bound = W.error_bound(dyb, xq, exact)
                got = W.widen_bf16(bits(model[n].weight.grad))
                assert np.all(np.abs(got - exact) <= bound), (step, n)
                # the unquantised input would give another gradient
                other = W.wgrad_exact(dyb, xb)
                assert np.any(np.abs(got - other) > W.error_bound(dyb, xb, other)), (step, n)
                if model[n].bias is not None:
                    torch.testing.assert_close(model[n].bias.grad.float(),
                                               dys[n].reshape(-1, dys[n].shape[-1]).float().sum(0),
                                               rtol=2e-2, atol=1e-3)
            units.step(0.4, 1.5)
            if step == 1:
                assert units.query()["mask"].tolist() == [1, 0]
            model.zero_grad(set_to_none=True)
    finally:
        quant.close()
        units.close()
    # closing restores the modules' own forward
    assert "forward" not in model["a"].__dict__
