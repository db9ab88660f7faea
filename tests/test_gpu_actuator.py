"""The recovery actuator (per-token fake quantisation switched by the
controller's mask) against its oracle, bit for bit, through the C ABI."""
import numpy as np
import pytest

from gpu_util import assert_step_matches, require_gpu
from oracle import fakequant as FQ

pytestmark = pytest.mark.gpu

COLS = [8, 16, 1000, 4096, 11008, 16384, 24]
ROWS = [3, 1, 7, 5, 2, 4, 0]


def activations(rng):
    out = []
    for r, c in zip(ROWS, COLS):
        x = rng.normal(size=(r, c)).astype(np.float32) * (10.0 ** rng.uniform(-6, 2, (r, 1)))
        if r >= 3:
            x[1] = 0.0                                   # an all-zero token
            x[2, ::5] = -0.0                             # signed zeros inside a token
            x[2, 3] = 1e4                                # an outlier
        out.append(FQ.f32_to_bf16(x.astype(np.float32)))
    return out


def to_device(torch, a):
    t = torch.from_numpy(a.view(np.int16).copy()).to("cuda")
    assert t.data_ptr() % 16 == 0
    return t


@pytest.mark.parametrize("fmts", [(1, 0), (1, 3), (2, 0), (4, 2), (3, 1), (0, 0), (5, 0), (1, 5)])
@pytest.mark.parametrize("inplace", [False, True])
def test_actuator_matches_oracle(fmts, inplace):
    torch = require_gpu()
    from paper_2606_00539_amd import Actuator

    rng = np.random.default_rng(sum(fmts) * 7 + inplace)
    acts = activations(rng)
    U = len(acts)
    mask = (rng.random(U) < 0.5).astype(np.uint8)
    d_in = [to_device(torch, a) for a in acts]
    d_out = d_in if inplace else [torch.full_like(t, 0x5555) for t in d_in]
    d_mask = torch.from_numpy(mask).to("cuda")
    segs = [(i, o, a.shape[0], a.shape[1], b) for b, (i, o, a) in enumerate(zip(d_in, d_out, acts))]
    with Actuator(segs, U) as act:
        info = act.info()
        assert info["rows"] == sum(ROWS)
        act.apply(d_mask, *fmts)
        torch.cuda.synchronize()
    want = FQ.actuate(acts, mask, *fmts)
    for b, (o, w) in enumerate(zip(d_out, want)):
        got = o.cpu().numpy().view(np.uint16).reshape(w.shape)
        bad = np.argwhere(got != w)
        assert bad.size == 0, f"unit {b} fmt {fmts}: {len(bad)} differ, first {bad[:3].tolist()}"


def test_actuator_follows_the_controller_mask():
    """Zero-copy: the controller's device mask drives the actuator directly."""
    torch = require_gpu()
    from paper_2606_00539_amd import GNMR_FMT_BF16, GNMR_FMT_E2M1, Actuator, Controller

    U = 6
    rng = np.random.default_rng(5)
    acts = [FQ.f32_to_bf16(rng.normal(size=(16, 4096)).astype(np.float32)) for _ in range(U)]
    d_in = [to_device(torch, a) for a in acts]
    norms = torch.ones(U, dtype=torch.float64, device="cuda")
    with Controller(U, 5, 2, 1, 0.0, np.zeros(U + 1), [], []) as ctl, \
            Actuator([(t, t, 16, 4096, b) for b, t in enumerate(d_in)], U) as act:
        for _ in range(6):
            ctl.step_from_norms(norms, 1.1, 1.5)
        norms[[1, 4]] = 9.0                        # two units spike -> recovery path
        ctl.step_from_norms(norms, 1.1, 1.5)
        dmask = ctl.device_outputs()["mask"]
        act.apply(dmask, GNMR_FMT_E2M1, GNMR_FMT_BF16)
        torch.cuda.synchronize()
        mask = ctl.query()["mask"]
    assert mask.tolist() == [0, 1, 0, 0, 1, 0]
    for b in range(U):
        got = d_in[b].cpu().numpy().view(np.uint16).reshape(16, 4096)
        want = acts[b] if mask[b] else FQ.fakequant_rows(acts[b], GNMR_FMT_E2M1)
        assert np.array_equal(got, want)


def test_actuator_int8_ties_and_rejects_unknown_formats():
    """INT8: a token whose amax is 127 has scale 1, so every x + 0.5 is an
    exact tie (to the even integer); formats outside 0..5 are refused."""
    torch = require_gpu()
    from paper_2606_00539_amd import GNMR_FMT_INT8, Actuator, GnmrError

    k = np.arange(0, 127, dtype=np.float32)
    row = np.concatenate([[127.0], k + 0.5, -(k + 0.5), k, [-127.0]]).astype(np.float32)
    row = np.pad(row, (0, (-row.size) % 8))
    x = FQ.f32_to_bf16(np.stack([row, row * np.float32(2.0 ** -20)]))
    assert np.array_equal(FQ.bf16_to_f32(x)[0], row)          # every value exact in bf16
    d = to_device(torch, x)
    d_mask = torch.zeros(1, dtype=torch.uint8, device="cuda")
    with Actuator([(d, d, 2, row.size, 0)], 1) as act:
        for bad in (-1, GNMR_FMT_INT8 + 1):
            with pytest.raises(GnmrError):
                act.apply(d_mask, bad, 0)
            with pytest.raises(GnmrError):
                act.apply(d_mask, 0, bad)
        act.apply(d_mask, GNMR_FMT_INT8, 0)
        torch.cuda.synchronize()
    got = d.cpu().numpy().view(np.uint16).reshape(x.shape)
    assert np.array_equal(got, FQ.fakequant_rows(x, GNMR_FMT_INT8))
    q = FQ.bf16_to_f32(got)[0][1:128]
    assert np.array_equal(q, np.where(k % 2 == 0, k, k + 1))    # ties to even


def test_actuator_segments_may_share_an_input():
    """Two units read one activation matrix out of place into two outputs
    (shared reads are not races), one in the low-cost and one in the recovery
    format."""
    torch = require_gpu()
    from paper_2606_00539_amd import Actuator

    rng = np.random.default_rng(9)
    a = FQ.f32_to_bf16(rng.normal(size=(6, 1000)).astype(np.float32))
    d_in = to_device(torch, a)
    outs = [torch.full_like(d_in, 0x5555) for _ in range(2)]
    d_mask = torch.tensor([0, 1], dtype=torch.uint8, device="cuda")
    with Actuator([(d_in, outs[0], 6, 1000, 0), (d_in, outs[1], 6, 1000, 1)], 2) as act:
        act.apply(d_mask, 1, 5)
        torch.cuda.synchronize()
    assert np.array_equal(outs[0].cpu().numpy().view(np.uint16).reshape(a.shape),
                          FQ.fakequant_rows(a, 1))
    assert np.array_equal(outs[1].cpu().numpy().view(np.uint16).reshape(a.shape),
                          FQ.fakequant_rows(a, 5))
    assert np.array_equal(d_in.cpu().numpy().view(np.uint16).reshape(a.shape), a)


MATRIX_CASES = [(5, 8), (37, 4096), (3, 4104), (2, 16384), (9, 1000), (0, 64), (1, 11008)]


@pytest.mark.parametrize("rows,cols", MATRIX_CASES)
@pytest.mark.parametrize("inplace", [False, True])
def test_actuate_matrix_matches_oracle(rows, cols, inplace):
    """The table-free entry: one matrix, both kernel shapes (a wavefront per
    row up to 4096 features, a workgroup per longer row), the mask entry of
    its unit choosing between two formats, bit-exact."""
    torch = require_gpu()
    from paper_2606_00539_amd import gnmr_actuate_matrix

    rng = np.random.default_rng(rows * 131 + cols + inplace)
    x = rng.normal(size=(rows, cols)).astype(np.float32) * (10.0 ** rng.uniform(-4, 2, (rows, 1)))
    if rows >= 3:
        x[1] = 0.0
        x[2, ::7] = -0.0
    a = FQ.f32_to_bf16(x.astype(np.float32))
    mask = torch.tensor([0, 1, 0], dtype=torch.uint8, device="cuda")
    for unit, fmts in ((0, (3, 5)), (1, (2, 5)), (2, (0, 1))):
        d_in = to_device(torch, a)
        d_out = d_in if inplace else torch.full_like(d_in, 0x5555)
        gnmr_actuate_matrix(d_in, d_out, rows, cols, mask, unit, *fmts)
        torch.cuda.synchronize()
        want = FQ.fakequant_rows(a, fmts[1] if unit == 1 else fmts[0])
        got = d_out.cpu().numpy().view(np.uint16).reshape(a.shape)
        assert np.array_equal(got, want), f"unit {unit} fmts {fmts}"
        if not inplace:
            assert np.array_equal(d_in.cpu().numpy().view(np.uint16).reshape(a.shape), a)


def test_quantized_inputs_follow_the_controller():
    """QuantizedInputs on three bf16 linear layers registered as units: before
    any step every layer takes the low-cost format; after a step that puts
    layer 1 in A_t, layer 1 takes the recovery format.  Outputs equal the
    layer applied to the oracle's quantised input, bit for bit; the input
    gradient is the straight-through one."""
    torch = require_gpu()
    import torch.nn.functional as F

    from paper_2606_00539_amd import GNMR_FMT_E2M1, GNMR_FMT_INT8
    from paper_2606_00539_amd.torch_units import QuantizedInputs, TorchUnits

    torch.manual_seed(0)
    layers = torch.nn.ModuleDict({f"l{i}": torch.nn.Linear(256, 64 * (i + 1), bias=i == 2)
                                  for i in range(3)}).to("cuda", torch.bfloat16)
    units = TorchUnits([(n + ".weight", m.weight) for n, m in layers.items()],
                       window=5, max_o=1, lock_len=1, eps=0.0,
                       unit_of=lambda name: name[:-len(".weight")])
    quant = QuantizedInputs(units, layers.items(), GNMR_FMT_E2M1, GNMR_FMT_INT8)

    def check(expect_fmt):
        for b, (n, m) in enumerate(layers.items()):
            x = (torch.randn(2, 9, 256, device="cuda") * (b + 1)).to(torch.bfloat16)
            x.requires_grad_(True)
            y = m(x)
            xb = x.detach().cpu().view(torch.int16).numpy().view(np.uint16).reshape(-1, 256)
            xq = torch.from_numpy(FQ.fakequant_rows(xb, expect_fmt[b]).view(np.int16)).to("cuda")
            xq = xq.view(torch.bfloat16).reshape(x.shape).requires_grad_(True)
            ref = F.linear(xq, m.weight, m.bias)
            assert torch.equal(y, ref), f"{n}: output differs"
            dy = torch.randn_like(y)
            y.backward(dy)
            ref.backward(dy)
            assert torch.equal(x.grad, xq.grad), f"{n}: input gradient is not straight through"

    try:
        check([GNMR_FMT_E2M1] * 3)
        norms = torch.ones(3, dtype=torch.float64, device="cuda")
        for _ in range(6):
            units.ctl.step_from_norms(norms, 1.1, 1.5)
        norms[1] = 9.0                                  # layer 1 spikes -> A_t = {1}
        units.ctl.step_from_norms(norms, 1.1, 1.5)
        assert units.query()["mask"].tolist() == [0, 1, 0]
        check([GNMR_FMT_E2M1, GNMR_FMT_INT8, GNMR_FMT_E2M1])
        with pytest.raises(TypeError):
            layers["l0"](torch.randn(4, 256, device="cuda"))     # fp32 input
    finally:
        quant.close()
        units.close()
    # hooks removed: the layer sees its input unchanged
    x = torch.randn(3, 256, device="cuda").to(torch.bfloat16)
    assert torch.equal(layers["l0"](x), F.linear(x, layers["l0"].weight))


def test_training_loop_with_controller_and_actuator():
    """A few SGD steps of a small SwiGLU stack in bf16 with the whole loop in
    place: each projection's input quantised per token by QuantizedInputs
    (E2M1 on the low-cost path, BF16 on the recovery path) from the mask of
    the previous controller step, the controller stepping over the .grad
    buffers (reallocated every step by zero_grad(set_to_none=True)), and the
    optimizer.  Every layer input the hooks produced is the oracle's
    quantisation of the layer's real input under that mask; every controller
    step matches the oracle fed with float64 norms of the stored gradients."""
    torch = require_gpu()
    import torch.nn.functional as F

    from oracle import Controller as Oracle
    from oracle import unit_norm
    from paper_2606_00539_amd import GNMR_FMT_BF16, GNMR_FMT_E2M1
    from paper_2606_00539_amd.torch_units import QuantizedInputs, TorchUnits, llama_linear_units

    torch.manual_seed(3)
    d, f = 64, 128
    model = torch.nn.ModuleDict({"layers": torch.nn.ModuleList([
        torch.nn.ModuleDict({"gate_proj": torch.nn.Linear(d, f, bias=False),
                             "up_proj": torch.nn.Linear(d, f, bias=False),
                             "down_proj": torch.nn.Linear(f, d, bias=False)})
        for _ in range(2)])}).to("cuda", torch.bfloat16)
    params = list(model.named_parameters())
    units = TorchUnits(params, max_o=2, lock_len=1, eps=1e-12, unit_of=llama_linear_units)
    U = len(units.unit_names)
    assert U == 6
    ora = Oracle(U, window=5, max_o=2, lock_len=1, eps=1e-12)
    seen = {}

    def capture(name):
        def pre(module, args):
            seen[name] = [args[0].detach().clone()]
        return pre

    def after(name):
        def post(module, args, out):
            seen[name].append(args[0].detach().clone())
        return post

    named = [(n, m) for n, m in model.named_modules() if n in units.unit_names]
    hooks = [m.register_forward_pre_hook(capture(n)) for n, m in named]
    quant = QuantizedInputs(units, named, GNMR_FMT_E2M1, GNMR_FMT_BF16)
    hooks += [m.register_forward_hook(after(n)) for n, m in named]
    opt = torch.optim.SGD(model.parameters(), lr=0.5)

    def bits(t):
        return t.view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1, t.shape[-1])

    mask_prev = np.zeros(U, np.uint8)
    recovered = 0
    try:
        for t in range(1, 9):
            x = torch.randn(2, 16, d, device="cuda").to(torch.bfloat16)
            h = x
            for blk in model["layers"]:
                h = h + blk["down_proj"](F.silu(blk["gate_proj"](h)) * blk["up_proj"](h))
            loss = (h.float() ** 2).mean()
            loss.backward()
            for b, u in enumerate(units.unit_names):
                orig, used = seen[u]
                fmt = GNMR_FMT_BF16 if mask_prev[b] else GNMR_FMT_E2M1
                assert np.array_equal(bits(used), FQ.fakequant_rows(bits(orig), fmt)), \
                    f"t={t} {u}: the layer did not see its input in format {fmt}"
            units.step(0.9, 1.5)                      # alpha < 1: every unit is a candidate
            out = units.query()
            norms = [unit_norm([(bits(p.grad).ravel(), 1)]) for p in units.params]
            assert_step_matches(out, ora.step(norms, 0.9, 1.5), rtol=1e-5, what=f"t={t}")
            assert out["mask"].sum() <= 2
            recovered += int(out["mask"].sum())
            mask_prev = out["mask"].copy()
            opt.step()
            opt.zero_grad(set_to_none=True)
        assert recovered > 0
    finally:
        for hk in hooks:
            hk.remove()
        quant.close()
        units.close()


def test_actuator_fullsize_bench_configuration():
    """The benchmark's launch configuration: one actuator over the saved
    activations of the 7 projections of 32 LLaMA-2-7B layers at 4,096 tokens
    (224 units, 9.33 GB, in place), 8 units on the recovery path (BF16), the
    rest on E2M1.  Sampled rows of every unit kind are checked bit for bit
    against the oracle; every row is checked against properties that hold at
    any size (recovery rows untouched, signs kept, magnitudes within the row's
    largest one, the largest one kept)."""
    torch = require_gpu()
    from paper_2606_00539_amd import GNMR_FMT_BF16, GNMR_FMT_E2M1, Actuator

    tokens, U = 4096, 32 * 7
    cols = [4096] * 6 + [11008]
    shapes = [(tokens, cols[b % 7]) for b in range(U)]
    total = sum(r * c for r, c in shapes)
    gen = torch.Generator(device="cuda").manual_seed(7)
    buf = torch.randn(total, dtype=torch.float32, device="cuda", generator=gen).to(torch.bfloat16)
    segs, offs, off = [], [], 0
    for b, (r, c) in enumerate(shapes):
        p = buf.data_ptr() + 2 * off
        segs.append((p, p, r, c, b))
        offs.append(off)
        off += r * c
    mask = np.zeros(U, np.uint8)
    rec = np.random.default_rng(0).choice(U, 8, replace=False)
    mask[rec] = 1
    rng = np.random.default_rng(1)
    picks = [(b, int(r)) for b in sorted(set(rng.choice(U, 24, replace=False)) | set(rec[:2]) |
                                         {0, U - 1})
             for r in (0, tokens - 1, *rng.choice(tokens, 2, replace=False))]

    def row(t, b, r):
        c = shapes[b][1]
        return t[offs[b] + r * c: offs[b] + (r + 1) * c]

    before = {(b, r): row(buf, b, r).view(torch.int16).cpu().numpy().view(np.uint16)
              for b, r in picks}
    orig = buf.clone()
    with Actuator(segs, U) as act:
        act.apply(torch.from_numpy(mask).to("cuda"), GNMR_FMT_E2M1, GNMR_FMT_BF16)
        torch.cuda.synchronize()
    for b, r in picks:
        got = row(buf, b, r).view(torch.int16).cpu().numpy().view(np.uint16)
        fmt = GNMR_FMT_BF16 if mask[b] else GNMR_FMT_E2M1
        want = FQ.fakequant_rows(before[(b, r)][None, :], fmt)[0]
        assert np.array_equal(got, want), f"unit {b} row {r}"
    for b, (r, c) in enumerate(shapes):
        x = orig[offs[b]:offs[b] + r * c].view(r, c).float()
        y = buf[offs[b]:offs[b] + r * c].view(r, c).float()
        if mask[b]:
            assert torch.equal(x, y), f"unit {b}: a recovery-path row changed"
            continue
        amax = x.abs().amax(dim=1, keepdim=True)
        assert bool(((y == 0) | (torch.sign(y) == torch.sign(x))).all()), f"unit {b}: sign"
        assert bool((y.abs() <= amax * (1 + 2.0 ** -7)).all()), f"unit {b}: magnitude"
        ymax = y.abs().amax(dim=1, keepdim=True)
        assert bool(((ymax - amax).abs() <= amax * 2.0 ** -7).all()), f"unit {b}: row maximum"
    del orig, buf
