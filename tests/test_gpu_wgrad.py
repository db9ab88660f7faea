"""Parity of the producer-fused gradient pass: the weight-gradient GEMM with
the sum of squares in its epilogue (gnmr_wgrad_sumsq), and the controller
step fed by its tile partials (gnmr_step_from_partials).

Bars (oracle/wgrad.py states the readings):
  * integer operands whose every partial sum is exact in fp32 and bf16: dw
    bit-exact against the oracle, over several tiles and ragged edges in all
    three dimensions;
  * random bf16 operands: every dw element within error_bound() of the
    float64 product, and each tile's sum of squares equal to the float64 sum
    of squares of the dw values the kernel stored, within the fp32
    summation bound (264 additions of non-negative terms: 264 * 2^-24);
  * full size (13B layer shapes, 4096 tokens): sampled dw elements, computed
    one by one by the oracle, and sampled tiles;
  * controller: masks, locks and counters bit-exact against the oracle
    controller fed with the oracle's norms, and against gnmr_step (K1) over
    the same stored gradients.
"""
import sys

import numpy as np
import pytest

from gpu_util import assert_step_matches, require_gpu
from oracle import Controller as Oracle
from oracle import wgrad as W
from synth import wgrad as SW

pytestmark = pytest.mark.gpu

SS_RTOL = 264 * 2.0 ** -24


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")


def run_wgrad(torch, dy_bits, x_bits, dw=None, ss=None):
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq

    T, M = dy_bits.shape
    N = x_bits.shape[1]
    d_dy, d_x = to_dev(torch, dy_bits), to_dev(torch, x_bits)
    if dw is None:
        dw = torch.full((M, N), 0x5555, dtype=torch.int16, device="cuda")   # unwritten marker
    nt = gnmr_wgrad_num_tiles(M, N)
    if ss is None:
        ss = torch.full((nt,), float("nan"), dtype=torch.float32, device="cuda")
    gnmr_wgrad_sumsq(d_dy, d_x, dw, T, M, N, ss)
    torch.cuda.synchronize()
    return dw.cpu().numpy().view(np.uint16), ss.cpu().numpy()


@pytest.mark.parametrize("M,N,T", [(256, 256, 64), (264, 520, 70), (520, 776, 130),
                                   (8, 8, 1), (16, 2056, 33), (1032, 264, 200)])
def test_integer_operands_bit_exact(M, N, T):
    torch = require_gpu()
    say(f"wgrad integer M={M} N={N} T={T}")
    dy, x = SW.small_integer_operands(M * 7 + N + T, T, M, N, vmax=1)
    dw, ss = run_wgrad(torch, dy, x)
    exact = W.wgrad_exact(dy, x)
    want = W.bf16_rne(exact)
    bad = np.argwhere(dw != want)
    assert bad.size == 0, f"dw differs at {bad[:8].tolist()}"
    ref = W.tile_sumsq(want)
    assert ss.shape == ref.shape
    np.testing.assert_allclose(ss, ref, rtol=SS_RTOL, atol=0)


def test_empty_batch_gives_zero_gradient():
    torch = require_gpu()
    dy = np.zeros((0, 264), np.uint16)
    x = np.zeros((0, 520), np.uint16)
    dw, ss = run_wgrad(torch, dy, x)
    assert np.all(dw == 0) and np.all(ss == 0.0)


def test_single_token_outer_product():
    torch = require_gpu()
    dy, x = SW.operands(5, 1, 0, tokens=1, out_f=272, in_f=328)
    dw, _ = run_wgrad(torch, dy, x)
    # one product per element: exact in fp32, so one rounding to bf16
    assert np.array_equal(dw, W.bf16_rne(W.wgrad_exact(dy, x)))


@pytest.mark.parametrize("M,N,T", [(576, 776, 1000), (256, 512, 4096), (200, 264, 65)])
def test_random_operands_within_bound(M, N, T):
    torch = require_gpu()
    say(f"wgrad random M={M} N={N} T={T}")
    dy, x = SW.operands(1, 1, M + N, tokens=T, out_f=M, in_f=N)
    dw, ss = run_wgrad(torch, dy, x)
    exact = W.wgrad_exact(dy, x)
    bound = W.error_bound(dy, x, exact)
    err = np.abs(W.widen_bf16(dw) - exact)
    bad = np.argwhere(err > bound)
    assert bad.size == 0, f"dw outside the bound at {bad[:8].tolist()}"
    # the epilogue sums the squares of exactly what it stored
    np.testing.assert_allclose(ss, W.tile_sumsq(dw), rtol=SS_RTOL, atol=0)
    # and the unit norm is within the bound's reach of the oracle's
    # (triangle inequality: | ||q|| - ||r|| | <= ||q - r|| <= ||2 bound||)
    n_gpu = np.sqrt(np.sum(ss.astype(np.float64)))
    n_ref = W.unit_norm(W.bf16_rne(exact))
    assert abs(n_gpu - n_ref) <= 2 * np.sqrt(np.sum(bound * bound)) + SS_RTOL * n_ref


def test_output_buffer_fully_written_and_nothing_else():
    torch = require_gpu()
    M, N, T = 264, 520, 70
    dy, x = SW.operands(2, 1, 9, tokens=T, out_f=M, in_f=N)
    guard = torch.full((M * N + 4096,), 0x5555, dtype=torch.int16, device="cuda")
    dw_view = guard[:M * N].view(M, N)
    run_wgrad(torch, dy, x, dw=dw_view)
    tail = guard[M * N:].cpu().numpy()
    assert np.all(tail == 0x5555), "K5 wrote past the end of dw"
    assert not np.any(dw_view.cpu().numpy().view(np.uint16) == 0x5555)


@pytest.mark.parametrize("M,N", [(13824, 5120), (5120, 13824)])
def test_fullsize_sampled(M, N):
    torch = require_gpu()
    T = 4096
    say(f"wgrad full size M={M} N={N} T={T}")
    dy, x = SW.operands(0, 1, 4, tokens=T, out_f=M, in_f=N)
    dw, ss = run_wgrad(torch, dy, x)
    assert ss.size == W.num_tiles(M, N)
    rng = np.random.default_rng(M)
    rows = rng.choice(M, 24, replace=False)
    cols = rng.choice(N, 24, replace=False)
    exact = W.wgrad_exact(dy[:, rows], x[:, cols])
    bound = W.error_bound(dy[:, rows], x[:, cols], exact)
    err = np.abs(W.widen_bf16(dw[np.ix_(rows, cols)]) - exact)
    assert np.all(err <= bound)
    tn = -(-N // 256)
    for tile in rng.choice(ss.size, 4, replace=False):
        a, b = divmod(int(tile), tn)
        blk = dw[a * 256:(a + 1) * 256, b * 256:(b + 1) * 256]
        np.testing.assert_allclose(ss[tile], W.tile_sumsq(blk)[0], rtol=SS_RTOL, atol=0)


@pytest.mark.parametrize("count", [5, 20])
def test_batched_matches_single_problem_calls(count):
    """One launch over several problems (and more than one launch past 16
    problems): every dw bit-identical to the oracle on integer operands and
    to the single-problem entry, tile sums at the concatenated offsets."""
    torch = require_gpu()
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    shapes = [(264, 520, 70), (8, 8, 1), (1032, 264, 200), (16, 2056, 33), (512, 256, 0)]
    shapes = [shapes[i % len(shapes)] for i in range(count)]
    say(f"wgrad batched, {count} problems")
    ops = [SW.small_integer_operands(11 + i, T, M, N) for i, (M, N, T) in enumerate(shapes)]
    dev = [(to_dev(torch, dy), to_dev(torch, x),
            torch.full((M, N), 0x5555, dtype=torch.int16, device="cuda"))
           for (dy, x), (M, N, T) in zip(ops, shapes)]
    tiles = [gnmr_wgrad_num_tiles(M, N) for M, N, _ in shapes]
    off = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    ss = torch.full((int(off[-1]),), float("nan"), dtype=torch.float32, device="cuda")
    gnmr_wgrad_sumsq_batched([(a, b, c, T, M, N) for (a, b, c), (M, N, T) in zip(dev, shapes)],
                             ss)
    torch.cuda.synchronize()
    ss = ss.cpu().numpy()
    for i, ((dy, x), (M, N, T), (_, _, c)) in enumerate(zip(ops, shapes, dev)):
        dw = c.cpu().numpy().view(np.uint16)
        want = W.bf16_rne(W.wgrad_exact(dy, x))
        assert np.array_equal(dw, want), f"problem {i}"
        np.testing.assert_allclose(ss[off[i]:off[i + 1]], W.tile_sumsq(want), rtol=SS_RTOL,
                                   atol=0, err_msg=f"problem {i}")
        dw1, ss1 = run_wgrad(torch, dy, x)
        assert np.array_equal(dw1, dw) and np.array_equal(ss1, ss[off[i]:off[i + 1]])


def test_batched_problems_may_share_operands():
    """Four problems read one input x (as q, k and v do) and write four
    gradients; a fifth reuses the first one's dy.  Shared reads pass the
    overlap checks, and every result is the oracle's, bit for bit on integer
    operands."""
    torch = require_gpu()
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    T, N = 130, 264
    outs = [264, 72, 72, 520]
    say("wgrad batched with shared operands")
    _, x = SW.small_integer_operands(31, T, 8, N)
    dys = [SW.small_integer_operands(32 + i, T, M, 8)[0] for i, M in enumerate(outs)]
    d_x = to_dev(torch, x)
    d_dy = [to_dev(torch, d) for d in dys]
    dws = [torch.full((M, N), 0x5555, dtype=torch.int16, device="cuda") for M in outs]
    # problem 4 reuses problem 0's dy against a second input of its own
    _, x2 = SW.small_integer_operands(36, T, 8, 136)
    d_x2 = to_dev(torch, x2)
    dw4 = torch.full((outs[0], 136), 0x5555, dtype=torch.int16, device="cuda")
    probs = [(d_dy[i], d_x, dws[i], T, M, N) for i, M in enumerate(outs)]
    probs.append((d_dy[0], d_x2, dw4, T, outs[0], 136))
    tiles = [gnmr_wgrad_num_tiles(M, N) for M in outs] + [gnmr_wgrad_num_tiles(outs[0], 136)]
    off = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    ss = torch.full((int(off[-1]),), float("nan"), dtype=torch.float32, device="cuda")
    gnmr_wgrad_sumsq_batched(probs, ss)
    torch.cuda.synchronize()
    ss = ss.cpu().numpy()
    wants = [W.bf16_rne(W.wgrad_exact(d, x)) for d in dys] + [W.bf16_rne(W.wgrad_exact(dys[0], x2))]
    for i, (got, want) in enumerate(zip(dws + [dw4], wants)):
        assert np.array_equal(got.cpu().numpy().view(np.uint16), want), f"problem {i}"
        np.testing.assert_allclose(ss[off[i]:off[i + 1]], W.tile_sumsq(want), rtol=SS_RTOL,
                                   atol=0, err_msg=f"problem {i}")


def small_layer():
    return SW.WgradLayer("small-layer", ((512, 512), (512, 512), (512, 512), (512, 512),
                                         (1376, 512), (1376, 512), (512, 1376)), tokens=256)


def test_controller_from_partials_matches_oracle_and_k1():
    torch = require_gpu()
    from paper_2606_00539_amd import Controller, gnmr_wgrad_num_tiles

    L = small_layer()
    U = L.num_units
    steps, window, max_o, lock_len, eps = 14, 5, 2, 3, 1e-12
    numel = [o * i for o, i in L.shapes]
    off = np.concatenate([[0], np.cumsum(numel)]).astype(np.int64)
    grads = torch.zeros(int(off[-1]), dtype=torch.int16, device="cuda")
    tiles = [gnmr_wgrad_num_tiles(o, i) for o, i in L.shapes]
    part_off = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    parts = torch.zeros(int(part_off[-1]), dtype=torch.float32, device="cuda")
    ptrs = [grads.data_ptr() + 2 * int(off[b]) for b in range(U)]
    fused = Controller(U, window, max_o, lock_len, eps, np.arange(U + 1), numel, [1] * U, ptrs)
    fused.bind_partials(part_off)
    k1 = Controller(U, window, max_o, lock_len, eps, np.arange(U + 1), numel, [1] * U, ptrs)
    ora = Oracle(U, window=window, max_o=max_o, lock_len=lock_len, eps=eps)
    from paper_2606_00539_amd import gnmr_wgrad_sumsq
    try:
        for t in range(1, steps + 1):
            alpha, beta = (1.5 if t == 1 else 1.1), 1.5
            norms = np.zeros(U)
            for b, (o, i) in enumerate(L.shapes):
                dy, x = SW.operands(L.seed, t, b, L.tokens, o, i, dy_scale=L.dy_scale(t, b))
                d_dy, d_x = to_dev(torch, dy), to_dev(torch, x)
                dw = grads[int(off[b]):int(off[b + 1])]
                gnmr_wgrad_sumsq(d_dy, d_x, dw, L.tokens, o, i,
                                 parts[int(part_off[b]):int(part_off[b + 1])])
                norms[b] = W.unit_norm(W.bf16_rne(W.wgrad_exact(dy, x)))
            fused.step_from_partials(parts, alpha, beta)
            k1.step(alpha, beta)
            ref = ora.step(norms, alpha, beta)
            # the scenario keeps every decision clear of its threshold
            g, d = ref.gnmr / alpha, ref.dgnmr / beta
            assert np.all(np.abs(g - 1) > 1e-3) and np.all(np.abs(d - 1) > 1e-3), f"t={t}"
            out_f, out_k = fused.query(), k1.query()
            # bf16 rounding of the fp32 accumulation moves a norm by far less
            # than 1e-3 relative; decisions must agree exactly
            assert_step_matches(out_f, ref, rtol=1e-3, what=f"fused t={t}")
            assert_step_matches(out_k, ref, rtol=1e-3, what=f"k1 t={t}")
            np.testing.assert_allclose(out_f["norm"], out_k["norm"], rtol=1e-5, atol=0,
                                       err_msg=f"t={t}: fused vs K1 norms of the same gradient")
            say(f"  t={t} ok: {out_f['stats']}")
        assert out_f["stats"]["t"] == steps
    finally:
        fused.close()
        k1.close()


def test_partials_binding_errors():
    torch = require_gpu()
    from paper_2606_00539_amd import Controller, GnmrError

    with Controller(3, 5, 1, 2, 0.0, [0, 1, 2, 3], [8, 8, 8], [1, 1, 1]) as ctl:
        parts = torch.zeros(4, dtype=torch.float32, device="cuda")
        with pytest.raises(GnmrError, match="GNMR_E_STATE"):
            ctl.step_from_partials(parts, 1.5, 1.5)
        for bad in ([1, 1, 2, 4], [0, 3, 2, 4], [0, 1, 2, -1]):
            with pytest.raises(GnmrError, match="GNMR_E_INVALID"):
                ctl.bind_partials(bad)
        with pytest.raises(ValueError):
            ctl.bind_partials([0, 1, 4])
        ctl.bind_partials([0, 1, 3, 4])
        with pytest.raises(GnmrError, match="GNMR_E_INVALID"):
            ctl.step_from_partials(parts, -1.0, 1.5)
        parts.copy_(torch.tensor([4.0, 1.0, 3.0, 9.0]))
        ctl.step_from_partials(parts, 1.5, 1.5)
        out = ctl.query()
        np.testing.assert_allclose(out["norm"], [2.0, 2.0, 3.0], rtol=1e-15)


def test_layer_fullsize_batched_step_matches_oracle():
    """The benchmark's launch configuration: the seven weight-gradient GEMMs
    of a LLaMA-2-13B layer at 4,096 tokens in one batched launch, then the
    controller step from the tile partials, for two steps.  Sampled dw
    elements are computed one by one by the oracle; sampled tiles and every
    unit norm are checked against float64 sums over the stored gradient; the
    step's decisions against the oracle controller."""
    torch = require_gpu()
    from paper_2606_00539_amd import Controller, gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    L = SW.llama2_13b_layer(4096)
    U, T = L.num_units, L.tokens
    numel = [o * i for o, i in L.shapes]
    off = np.concatenate([[0], np.cumsum(numel)]).astype(np.int64)
    grads = torch.empty(int(off[-1]), dtype=torch.int16, device="cuda")
    dws = [grads[int(off[b]):int(off[b + 1])].view(o, i) for b, (o, i) in enumerate(L.shapes)]
    tiles = [gnmr_wgrad_num_tiles(o, i) for o, i in L.shapes]
    poff = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    parts = torch.full((int(poff[-1]),), float("nan"), dtype=torch.float32, device="cuda")
    ptrs = [d.data_ptr() for d in dws]
    ora = Oracle(U, window=5, max_o=2, lock_len=4, eps=1e-12)
    rng = np.random.default_rng(13)
    with Controller(U, 5, 2, 4, 1e-12, np.arange(U + 1), numel, [1] * U, ptrs) as ctl:
        ctl.bind_partials(poff)
        for t in (1, 2):
            say(f"wgrad 13B layer batched, step {t}")
            ops = [SW.operands(L.seed, t, b, T, o, i, dy_scale=L.dy_scale(t, b))
                   for b, (o, i) in enumerate(L.shapes)]
            dev = [(to_dev(torch, dy), to_dev(torch, x)) for dy, x in ops]
            gnmr_wgrad_sumsq_batched([(a, c, dws[b], T, o, i) for b, ((a, c), (o, i))
                                      in enumerate(zip(dev, L.shapes))], parts)
            alpha, beta = (1.5 if t == 1 else 1.1), 1.5
            ctl.step_from_partials(parts, alpha, beta)
            out = ctl.query()
            ss = parts.cpu().numpy()
            norms = np.zeros(U)
            for b, ((dy, x), (o, i)) in enumerate(zip(ops, L.shapes)):
                dw = dws[b].cpu().numpy().view(np.uint16)
                rows = rng.choice(o, 16, replace=False)
                cols = rng.choice(i, 16, replace=False)
                exact = W.wgrad_exact(dy[:, rows], x[:, cols])
                bound = W.error_bound(dy[:, rows], x[:, cols], exact)
                err = np.abs(W.widen_bf16(dw[np.ix_(rows, cols)]) - exact)
                assert np.all(err <= bound), f"t={t} unit {b}: dw outside the bound"
                ts = ss[poff[b]:poff[b + 1]]
                tn = -(-i // 256)
                for tile in rng.choice(ts.size, 3, replace=False):
                    a, c = divmod(int(tile), tn)
                    blk = dw[a * 256:(a + 1) * 256, c * 256:(c + 1) * 256]
                    np.testing.assert_allclose(ts[tile], W.tile_sumsq(blk)[0], rtol=SS_RTOL,
                                               atol=0, err_msg=f"t={t} unit {b} tile {tile}")
                norms[b] = W.unit_norm(dw)
                del dw
            ref = ora.step(norms, alpha, beta)
            g, d = ref.gnmr / alpha, ref.dgnmr / beta
            assert np.all(np.abs(g - 1) > 1e-3) and np.all(np.abs(d - 1) > 1e-3), f"t={t}"
            # fp32 tile sums (each within 264 roundings) against the float64
            # norm of the same stored values: relative 264 * 2^-24 / 2 on n,
            # at most twice that on a ratio of two norms
            assert_step_matches(out, ref, rtol=2 * SS_RTOL, what=f"13B layer t={t}")
            assert out["stats"]["t"] == t


def _tiny_block(torch, seed):
    """Seven bias-free bf16 projections shaped like a small decoder layer,
    each used once per forward."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    names = ("q", "k", "v", "o", "gate", "up", "down")
    shapes = ((256, 256), (256, 256), (256, 256), (256, 256), (688, 256), (688, 256),
              (256, 688))
    mods = torch.nn.ModuleDict()
    for n, (o, i) in zip(names, shapes):
        lin = torch.nn.Linear(i, o, bias=False)
        with torch.no_grad():
            lin.weight.copy_(torch.randn(o, i, generator=g) * (1.0 / i ** 0.5))
        mods[n] = lin
    return mods.to(device="cuda", dtype=torch.bfloat16)


def _block_forward(m, x, q_gain=1.0):
    a = m["q"](x * q_gain) + m["k"](x) + m["v"](x)
    h = m["o"](a)
    return m["down"](m["gate"](h) * m["up"](h))


def test_fused_wgrad_units_in_autograd_match_torch_and_k1():
    """FusedWgradUnits routes a model's linear layers through K5 in backward:
    the weight gradients agree with torch's own backward within two bf16
    roundings, the controller step from the tile partials makes the same
    decisions as the K1 step (TorchUnits) over the same stored gradients, and
    a second micro-batch accumulates into the stored gradients."""
    import copy

    torch = require_gpu()
    from paper_2606_00539_amd.torch_units import FusedWgradUnits, TorchUnits

    fused_m = _tiny_block(torch, 7)
    ref_m = copy.deepcopy(fused_m)
    fused = FusedWgradUnits(list(fused_m.items()), max_o=2, lock_len=2)
    k1 = TorchUnits(list(fused_m.named_parameters()), max_o=2, lock_len=2)
    ora = Oracle(7, window=5, max_o=2, lock_len=2, eps=1e-12)
    g = torch.Generator(device="cpu").manual_seed(3)
    try:
        for t in range(1, 9):
            say(f"fused autograd step {t}")
            x = (torch.randn(200, 256, generator=g)).to("cuda", torch.bfloat16)
            for model in (fused_m, ref_m):
                model.zero_grad(set_to_none=True)
                # a x5 spike in the q projection's gradient at step 6
                y = _block_forward(model, x, q_gain=5.0 if t == 6 else 1.0)
                loss = y.float().square().mean()
                loss.backward()
            # torch's own backward of the same model: dW within two bf16 roundings
            for n in fused_m:
                a = fused_m[n].weight.grad.float()
                b = ref_m[n].weight.grad.float()
                tol = 2.0 ** -7 * b.abs() + 1e-3 * b.abs().max()
                assert bool(((a - b).abs() <= tol).all()), f"t={t} {n}: dW differs from torch"
            alpha, beta = (1.5 if t == 1 else 1.1), 1.5
            fused.step(alpha, beta)
            k1.step(alpha, beta)
            out_f, out_k = fused.query(), k1.query()
            norms = np.array([W.unit_norm(fused_m[n].weight.grad.view(torch.int16).cpu().numpy()
                                          .view(np.uint16)) for n in fused_m])
            ref = ora.step(norms, alpha, beta)
            gm, dm = ref.gnmr / alpha, ref.dgnmr / beta
            assert np.all(np.abs(gm - 1) > 1e-4) and np.all(np.abs(dm - 1) > 1e-4), f"t={t}"
            r = np.sort(ref.risk[ref.risk > 1.0])[::-1]
            if r.size > 2:      # the cap binds: the 2nd and 3rd risks are clearly apart
                assert (r[1] - r[2]) / r[1] > 1e-4, f"t={t}: near-tie at the cut"
            assert_step_matches(out_f, ref, rtol=2 * SS_RTOL, what=f"fused t={t}")
            assert_step_matches(out_k, ref, rtol=1e-5, what=f"k1 t={t}")
            if t == 6:
                assert out_f["mask"][0] == 1, "the q spike must send q to the recovery path"
        # gradient accumulation: a second micro-batch before the step adds to
        # the stored gradients in place, as torch's own backward would, and
        # the step's norms are those of the accumulated gradients
        # (a [batch, sequence, features] micro-batch: 2 x 68 tokens)
        x2 = torch.randn(2, 68, 256, generator=g).to("cuda", torch.bfloat16)
        for model in (fused_m, ref_m):
            _block_forward(model, x2).float().square().mean().backward()
        for n in fused_m:
            a = fused_m[n].weight.grad.float()
            b = ref_m[n].weight.grad.float()
            tol = 2.0 ** -6 * b.abs() + 2e-3 * b.abs().max()
            assert bool(((a - b).abs() <= tol).all()), f"accumulated {n}: dW differs from torch"
        fused.step(1.1, 1.5)
        out_f = fused.query()
        norms = np.array([W.unit_norm(fused_m[n].weight.grad.view(torch.int16).cpu().numpy()
                                      .view(np.uint16)) for n in fused_m])
        np.testing.assert_allclose(out_f["norm"], norms, rtol=SS_RTOL, atol=0)
        # a layer that did not run since the last step is refused, not stale
        with pytest.raises(RuntimeError, match="did not run"):
            fused.step(1.1, 1.5)
    finally:
        fused.close()
        k1.close()


def test_fused_layer_step_captured_in_a_graph_replays_like_eager():
    """The batched K5 launch and the step from its partials, captured once in
    a HIP graph and replayed: with fresh operands copied in between replays
    (eager work and synchronisations in between), every replay's gradients,
    masks, locks and ratios are bit-identical to the same step run eagerly."""
    torch = require_gpu()
    from paper_2606_00539_amd import Controller, gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    L = small_layer()
    U, T = L.num_units, L.tokens
    steps, capture_at = 10, 3
    numel = [o * i for o, i in L.shapes]
    tiles = [gnmr_wgrad_num_tiles(o, i) for o, i in L.shapes]
    poff = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    dys = [torch.empty((T, o), dtype=torch.int16, device="cuda") for o, _ in L.shapes]
    xs = [torch.empty((T, i), dtype=torch.int16, device="cuda") for _, i in L.shapes]

    def side_buffers():
        dws = [torch.empty((o, i), dtype=torch.int16, device="cuda") for o, i in L.shapes]
        parts = torch.empty(int(poff[-1]), dtype=torch.float32, device="cuda")
        return dws, parts

    def problems(dws):
        return [(dys[b], xs[b], dws[b], T, o, i) for b, (o, i) in enumerate(L.shapes)]

    def load(t):
        for b, (o, i) in enumerate(L.shapes):
            dy, x = SW.operands(L.seed, t, b, T, o, i, dy_scale=L.dy_scale(t, b))
            dys[b].copy_(torch.from_numpy(dy.view(np.int16)))
            xs[b].copy_(torch.from_numpy(x.view(np.int16)))
        torch.cuda.synchronize()

    (dws_e, parts_e), (dws_g, parts_g) = side_buffers(), side_buffers()
    mk = lambda: Controller(U, 5, 2, 3, 1e-12, np.zeros(U + 1, np.int64), [], [])
    with mk() as eager, mk() as graphed:
        eager.bind_partials(poff)
        graphed.bind_partials(poff)
        graph, side = torch.cuda.CUDAGraph(), torch.cuda.Stream()
        for t in range(1, steps + 1):
            say(f"fused graph t={t}")
            load(t)
            alpha = 1.5 if t == 1 else 1.1
            gnmr_wgrad_sumsq_batched(problems(dws_e), parts_e)
            eager.step_from_partials(parts_e, alpha, 1.5)
            if t < capture_at:
                gnmr_wgrad_sumsq_batched(problems(dws_g), parts_g)
                graphed.step_from_partials(parts_g, alpha, 1.5)
            else:
                if t == capture_at:
                    torch.cuda.synchronize()
                    with torch.cuda.stream(side):
                        with torch.cuda.graph(graph, stream=side):
                            gnmr_wgrad_sumsq_batched(problems(dws_g), parts_g, side)
                            graphed.step_from_partials(parts_g, 1.1, 1.5, side)
                    torch.cuda.synchronize()
                    assert graphed.query()["stats"]["t"] == capture_at - 1
                graph.replay()
            torch.cuda.synchronize()
            oe, og = eager.query(), graphed.query()
            for b in range(U):
                assert torch.equal(dws_e[b], dws_g[b]), f"t={t} unit {b}: dw"
            assert torch.equal(parts_e, parts_g), f"t={t}: tile partials"
            for k in ("mask", "lock", "norm", "gnmr", "dgnmr", "risk"):
                assert np.array_equal(oe[k], og[k]), f"t={t}: {k}"
            assert oe["stats"] == og["stats"], f"t={t}: stats"
        assert og["stats"]["t"] == steps


@pytest.mark.parametrize("M,N,T", [(264, 520, 70), (1032, 264, 200), (8, 8, 1)])
def test_accumulate_integer_operands_bit_exact(M, N, T):
    """accumulate = 1 on integer data whose sums stay exact: the stored
    gradient becomes bf16(old + dy^T x) bit for bit, tile sums of the result."""
    torch = require_gpu()
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    say(f"wgrad accumulate integer M={M} N={N} T={T}")
    dy, x = SW.small_integer_operands(M + 3 * N + T, T, M, N, vmax=1)
    rng = np.random.default_rng(M * N)
    old = W.bf16_rne(rng.integers(-8, 9, size=(M, N)).astype(np.float64))
    dw = to_dev(torch, old)
    ss = torch.full((gnmr_wgrad_num_tiles(M, N),), float("nan"), device="cuda")
    gnmr_wgrad_sumsq_batched([(to_dev(torch, dy), to_dev(torch, x), dw, T, M, N, 1)], ss)
    torch.cuda.synchronize()
    got = dw.cpu().numpy().view(np.uint16)
    want = W.bf16_rne(W.wgrad_accumulate_exact(old, dy, x))
    assert np.array_equal(got, want)
    np.testing.assert_allclose(ss.cpu().numpy(), W.tile_sumsq(want), rtol=SS_RTOL, atol=0)


def test_accumulate_random_operands_within_bound_and_mixed_batch():
    """Random operands: accumulated gradients inside error_bound_accumulate,
    tile sums of exactly what was stored; in one batched launch next to a
    non-accumulating problem, which still overwrites."""
    torch = require_gpu()
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    shapes = [(576, 776, 1000), (264, 520, 300)]
    ops = [SW.operands(4, 1, b, tokens=T, out_f=M, in_f=N) for b, (M, N, T) in enumerate(shapes)]
    olds = [W.bf16_rne(W.wgrad_exact(*SW.operands(4, 2, b, tokens=T, out_f=M, in_f=N)))
            for b, (M, N, T) in enumerate(shapes)]
    dws = [to_dev(torch, o) for o in olds]
    tiles = [gnmr_wgrad_num_tiles(M, N) for M, N, _ in shapes]
    off = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    ss = torch.full((int(off[-1]),), float("nan"), device="cuda")
    gnmr_wgrad_sumsq_batched([(to_dev(torch, dy), to_dev(torch, x), dws[b], T, M, N, 1 - b)
                              for b, ((dy, x), (M, N, T)) in enumerate(zip(ops, shapes))], ss)
    torch.cuda.synchronize()
    ss = ss.cpu().numpy()
    for b, ((dy, x), (M, N, T)) in enumerate(zip(ops, shapes)):
        got = dws[b].cpu().numpy().view(np.uint16)
        if b == 0:
            exact = W.wgrad_accumulate_exact(olds[b], dy, x)
            bound = W.error_bound_accumulate(olds[b], dy, x, exact)
        else:
            exact = W.wgrad_exact(dy, x)
            bound = W.error_bound(dy, x, exact)
        bad = np.argwhere(np.abs(W.widen_bf16(got) - exact) > bound)
        assert bad.size == 0, f"problem {b}: outside the bound at {bad[:8].tolist()}"
        np.testing.assert_allclose(ss[off[b]:off[b + 1]], W.tile_sumsq(got), rtol=SS_RTOL,
                                   atol=0, err_msg=f"problem {b}")


@pytest.mark.parametrize("M,N", [(13824, 5120), (5120, 13824)])
def test_accumulate_fullsize_sampled(M, N):
    """accumulate = 1 at a 13B layer's full shapes and 4,096 tokens: a stored
    gradient drawn on the host, then one micro-batch added by K5.  Sampled
    elements against the oracle's float64 old + dy^T x within
    error_bound_accumulate; sampled tile sums against float64 sums over the
    stored result."""
    torch = require_gpu()
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq_batched

    T = 4096
    say(f"wgrad accumulate full size {M}x{N}, {T} tokens")
    rng = np.random.default_rng(M + 7 * N)
    old = W.bf16_rne(rng.normal(scale=1e-3, size=(M, N)))
    dy, x = SW.operands(29, 2, 0, tokens=T, out_f=M, in_f=N)
    dw = to_dev(torch, old)
    ss = torch.full((gnmr_wgrad_num_tiles(M, N),), float("nan"), device="cuda")
    gnmr_wgrad_sumsq_batched([(to_dev(torch, dy), to_dev(torch, x), dw, T, M, N, 1)], ss)
    torch.cuda.synchronize()
    got = dw.cpu().numpy().view(np.uint16)
    rows = rng.choice(M, 24, replace=False)
    cols = rng.choice(N, 24, replace=False)
    exact = W.wgrad_accumulate_exact(old[np.ix_(rows, cols)], dy[:, rows], x[:, cols])
    bound = W.error_bound_accumulate(old[np.ix_(rows, cols)], dy[:, rows], x[:, cols], exact)
    err = np.abs(W.widen_bf16(got[np.ix_(rows, cols)]) - exact)
    assert np.all(err <= bound), f"{M}x{N}: accumulated dw outside the bound"
    ts = ss.cpu().numpy()
    tn = N // 256
    for tile in rng.choice(ts.size, 6, replace=False):
        a, c = divmod(int(tile), tn)
        blk = got[a * 256:(a + 1) * 256, c * 256:(c + 1) * 256]
        np.testing.assert_allclose(ts[tile], W.tile_sumsq(blk)[0], rtol=SS_RTOL, atol=0,
                                   err_msg=f"{M}x{N} tile {tile}")


def test_fused_wgrad_units_with_bias_and_unaligned_views():
    """A biased layer (bias gradient left to torch) fed a view that starts off
    a 16-byte boundary: the operand is copied to an aligned buffer, and dW,
    dx, the bias gradient and the step's norm match torch and the stored
    gradient."""
    import copy

    torch = require_gpu()
    from paper_2606_00539_amd.torch_units import FusedWgradUnits

    g = torch.Generator(device="cpu").manual_seed(9)
    lin = torch.nn.Linear(264, 136, bias=True)
    with torch.no_grad():
        lin.weight.copy_(torch.randn(136, 264, generator=g) * 0.05)
        lin.bias.copy_(torch.randn(136, generator=g))
    lin = lin.to("cuda", torch.bfloat16)
    ref = copy.deepcopy(lin)
    fused = FusedWgradUnits([("lin", lin)], max_o=1, lock_len=1)
    try:
        base = torch.randn(40 * 264 + 3, generator=g).to("cuda", torch.bfloat16)
        x = base[3:].view(40, 264)                     # 6 bytes past an aligned start
        assert x.data_ptr() % 16 != 0
        xa = x.detach().clone().requires_grad_(True)
        xb = x.detach().clone().requires_grad_(True)
        ya, yb = lin(xa), ref(xb)
        assert torch.equal(ya, yb), "the routed forward must be nn.Linear's"
        ya.float().square().sum().backward()
        yb.float().square().sum().backward()
        a, b = lin.weight.grad.float(), ref.weight.grad.float()
        assert bool(((a - b).abs() <= 2.0 ** -7 * b.abs() + 1e-3 * b.abs().max()).all())
        ga, gb = lin.bias.grad.float(), ref.bias.grad.float()
        assert bool(((ga - gb).abs() <= 2.0 ** -7 * gb.abs() + 1e-3 * gb.abs().max()).all())
        dxa, dxb = xa.grad.float(), xb.grad.float()
        assert bool(((dxa - dxb).abs() <= 2.0 ** -7 * dxb.abs() + 1e-3 * dxb.abs().max()).all())
        fused.step(1.5, 1.5)
        norm = fused.query()["norm"][0]
        want = W.unit_norm(lin.weight.grad.view(torch.int16).cpu().numpy().view(np.uint16))
        np.testing.assert_allclose(norm, want, rtol=SS_RTOL, atol=0)
    finally:
        fused.close()
