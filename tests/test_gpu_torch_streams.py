"""The PyTorch wrappers on a non-default stream: backward, the controller
step and the query all under `torch.cuda.stream(s)`, with the gradients
written on that stream.  The wrappers' default stream is torch's current one,
so the step is ordered after the backward that wrote the gradients; the
results must match the oracle fed with the stored gradients' norms, step
after step, for both the K1 path (TorchUnits) and the producer-fused path
(FusedWgradUnits)."""
import numpy as np
import pytest

from gpu_util import assert_step_matches, require_gpu
from oracle import Controller as Oracle
from oracle import unit_norm

pytestmark = pytest.mark.gpu


def grad_bits(p):
    import torch
    return p.grad.view(torch.int16).cpu().numpy().view(np.uint16).ravel()


@pytest.mark.parametrize("fused", [False, True])
def test_wrappers_on_a_side_stream_match_oracle(fused):
    torch = require_gpu()

    from paper_2606_00539_amd.torch_units import FusedWgradUnits, TorchUnits

    torch.manual_seed(11)
    shapes = {"q": (256, 512), "up": (768, 512), "down": (512, 768)}
    layers = torch.nn.ModuleDict({n: torch.nn.Linear(i, o, bias=False)
                                  for n, (o, i) in shapes.items()}).to("cuda", torch.bfloat16)
    if fused:
        units = FusedWgradUnits(list(layers.items()), max_o=1, lock_len=1, eps=1e-12)
    else:
        units = TorchUnits(layers.named_parameters(), max_o=1, lock_len=1, eps=1e-12,
                           unit_of=lambda n: n.split(".")[0])
    ora = Oracle(3, window=5, max_o=1, lock_len=1, eps=1e-12)
    side = torch.cuda.Stream()
    try:
        for t in range(1, 7):
            torch.cuda.synchronize()
            with torch.cuda.stream(side):
                # a large, slow-to-produce backward on the side stream: a step on
                # another stream would read stale or unwritten gradients
                x = torch.randn(4096, 512, device="cuda").to(torch.bfloat16)
                if t == 4:
                    x = x * 8                       # a spike: some unit triggers
                h = layers["q"](x)
                u = layers["up"](x)
                y = layers["down"](u)
                loss = (h.float() ** 2).mean() + (y.float() ** 2).mean()
                loss.backward()
                units.step(1.5, 1.5)
                out = units.query()
            norms = [unit_norm([(grad_bits(layers[n].weight), 1)]) for n in shapes]
            ref = ora.step(norms, 1.5, 1.5)
            # decisions far from their thresholds (fp32 against float64 norms)
            assert np.all(np.abs(ref.gnmr / 1.5 - 1) > 1e-4), t
            assert t <= 5 or np.all(np.abs(ref.dgnmr / 1.5 - 1) > 1e-4), t
            top = np.sort(ref.risk)[::-1]
            assert (top[0] - top[1]) > 1e-4 * top[0] or top[1] <= 1, t
            assert_step_matches(out, ref, rtol=1e-5, what=f"t={t}")
            layers.zero_grad(set_to_none=True)
    finally:
        units.close()
