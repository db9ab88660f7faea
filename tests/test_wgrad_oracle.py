"""Pins of the weight-gradient oracle (oracle/wgrad.py) against facts that
do not come from the oracle itself: brute force on tiny inputs, the rank-one
closed form of a single token, hand-derived bf16 bit patterns, the tiling's
element counts, and fp32 accumulations simulated in NumPy staying inside
error_bound()."""
import numpy as np
import pytest

from oracle import wgrad as W
from synth import wgrad as SW


def f32_to_bf16_trunc_exact(v):
    """bits of float32 values that are exactly bf16 (test helper)."""
    return (np.asarray(v, np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def test_wgrad_exact_matches_triple_loop():
    dy, x = SW.small_integer_operands(3, tokens=5, out_f=4, in_f=6, vmax=3)
    got = W.wgrad_exact(dy, x)
    a, b = W.widen_bf16(dy), W.widen_bf16(x)
    for o in range(4):
        for i in range(6):
            s = 0.0
            for t in range(5):
                s += a[t, o] * b[t, i]
            assert got[o, i] == s


def test_single_token_is_outer_product():
    dy = f32_to_bf16_trunc_exact([[0.5, -2.0, 3.0]])
    x = f32_to_bf16_trunc_exact([[1.0, 0.25]])
    got = W.wgrad_exact(dy, x)
    assert np.array_equal(got, np.array([[0.5, 0.125], [-2.0, -0.5], [3.0, 0.75]]))


def test_wgrad_is_transpose_sensitive():
    # dW[o][i] pairs dy's column o with x's column i: swapping operands
    # transposes the result
    dy, x = SW.small_integer_operands(4, tokens=7, out_f=3, in_f=5, vmax=2)
    assert np.array_equal(W.wgrad_exact(x, dy), W.wgrad_exact(dy, x).T)


@pytest.mark.parametrize("value,bits", [
    (1.0, 0x3F80), (-2.5, 0xC020), (0.0, 0x0000), (-0.0, 0x8000),
    (1 + 2 ** -8, 0x3F80),            # tie, even neighbour 1.0
    (1 + 3 * 2 ** -8, 0x3F82),        # tie between 0x3F81 and 0x3F82: even
    (1 + 2 ** -8 + 2 ** -30, 0x3F81),  # just above the tie
    (1 + 2 ** -8 - 2 ** -30, 0x3F80),  # just below the tie
    ((2 - 2 ** -7) * 2.0 ** 127, 0x7F7F),   # largest finite
    (3.5e38, 0x7F80),                 # overflow
    (2.0 ** -126, 0x0080),            # smallest normal
    (2.0 ** -133, 0x0001),            # smallest subnormal
    (2.0 ** -134, 0x0000),            # tie with zero: even
    (3 * 2.0 ** -135, 0x0001),
    (float("inf"), 0x7F80), (float("-inf"), 0xFF80),
])
def test_bf16_rne_bit_patterns(value, bits):
    assert int(W.bf16_rne(np.array([value]))[0]) == bits


def test_bf16_rne_nan_is_quiet_nan():
    assert int(W.bf16_rne(np.array([np.nan]))[0]) == 0x7FC0


def test_bf16_rne_keeps_representable_values():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 0x7F80, size=20000).astype(np.uint16)   # finite, non-negative
    bits = np.concatenate([bits, bits | np.uint16(0x8000)])
    assert np.array_equal(W.bf16_rne(W.widen_bf16(bits)), bits)


def test_bf16_rne_is_nearest():
    # against the two bf16 neighbours of each value, brute force
    rng = np.random.default_rng(1)
    v = rng.standard_normal(5000) * np.exp2(rng.integers(-20, 20, 5000))
    q = W.widen_bf16(W.bf16_rne(v))
    lo = W.widen_bf16(f32_to_bf16_trunc_exact(
        (np.abs(v).astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)))
    step = np.exp2(np.frexp(np.abs(v))[1] - 8.0)
    cands = np.stack([lo, lo + step])
    best = cands[np.argmin(np.abs(cands - np.abs(v)), axis=0), np.arange(v.size)]
    assert np.all(np.abs(np.abs(q) - np.abs(v)) <= np.abs(best - np.abs(v)))


@pytest.mark.parametrize("M,N", [(256, 256), (300, 256), (256, 520), (520, 776), (8, 8)])
def test_tile_sumsq_counts_every_element_once(M, N):
    one = np.full((M, N), 0x3F80, np.uint16)          # 1.0 everywhere
    ss = W.tile_sumsq(one)
    tm, tn = -(-M // 256), -(-N // 256)
    assert ss.size == W.num_tiles(M, N) == tm * tn
    for a in range(tm):
        for b in range(tn):
            rows = min(256, M - 256 * a)
            cols = min(256, N - 256 * b)
            assert ss[a * tn + b] == rows * cols       # row-major tile order, ragged edges
    assert ss.sum() == M * N


def test_tile_sumsq_tile_order_is_row_major():
    w = np.zeros((512, 768), np.uint16)
    w[300, 600] = 0x4000                             # 2.0 in tile (1, 2)
    ss = W.tile_sumsq(w)
    assert ss[1 * 3 + 2] == 4.0 and ss.sum() == 4.0


def test_unit_norm_closed_form():
    c = f32_to_bf16_trunc_exact([2.0 ** -10])[0]
    w = np.full((64, 48), c, np.uint16)
    w[::2] |= np.uint16(0x8000)
    assert W.unit_norm(w) == 2.0 ** -10 * np.sqrt(64 * 48)


def _fp32_accumulate(dy_bits, x_bits, order):
    """A NumPy stand-in for an fp32 accumulator: products are exact in fp32
    (8-bit significands), sums rounded to fp32 in the given token order."""
    a = W.widen_bf16(dy_bits).astype(np.float32)
    b = W.widen_bf16(x_bits).astype(np.float32)
    acc = np.zeros((a.shape[1], b.shape[1]), np.float32)
    for t in order:
        acc = (acc + np.outer(a[t], b[t]).astype(np.float32)).astype(np.float32)
    return acc


@pytest.mark.parametrize("order", ["forward", "reverse", "shuffled"])
def test_error_bound_covers_fp32_accumulation(order):
    dy, x = SW.operands(0, 1, 0, tokens=512, out_f=24, in_f=40, dy_scale=1e-3, x_scale=1.0)
    K = dy.shape[0]
    idx = {"forward": np.arange(K), "reverse": np.arange(K)[::-1],
           "shuffled": np.random.default_rng(2).permutation(K)}[order]
    acc = _fp32_accumulate(dy, x, idx)
    q = W.widen_bf16(W.bf16_rne(acc.astype(np.float64)))
    exact = W.wgrad_exact(dy, x)
    bound = W.error_bound(dy, x, exact)
    assert np.all(np.abs(q - exact) <= bound)
    # and the bound is not vacuous: far below the values themselves
    assert np.median(bound / np.abs(exact)) < 0.05


def test_error_bound_is_violated_by_a_dropped_token():
    # a plausible kernel mistake (one token row skipped) falls outside the bound
    dy, x = SW.operands(0, 1, 1, tokens=256, out_f=16, in_f=16)
    exact = W.wgrad_exact(dy, x)
    wrong = W.wgrad_exact(dy[1:], x[1:])
    q = W.widen_bf16(W.bf16_rne(wrong))
    assert np.any(np.abs(q - exact) > W.error_bound(dy, x, exact))


def test_operands_are_seeded_and_distinct():
    a = SW.operands(0, 1, 0, 8, 16, 24)
    b = SW.operands(0, 1, 0, 8, 16, 24)
    c = SW.operands(0, 2, 0, 8, 16, 24)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert not np.array_equal(a[0], c[0])
    assert a[0].shape == (8, 16) and a[1].shape == (8, 24)


def test_llama_layer_shapes():
    L = SW.llama2_13b_layer(4096)
    assert L.num_units == 7
    assert L.flops == 2 * 4096 * (4 * 5120 * 5120 + 3 * 13824 * 5120)
    assert L.grad_bytes == 2 * (4 * 5120 * 5120 + 3 * 13824 * 5120)


@pytest.mark.parametrize("order", ["forward", "shuffled"])
def test_accumulate_bound_covers_fp32_add_then_bf16(order):
    # a stored bf16 gradient plus an fp32 accumulation, added in fp32 and
    # rounded to bf16 once: inside error_bound_accumulate
    dy, x = SW.operands(0, 1, 2, tokens=384, out_f=24, in_f=40, dy_scale=1e-3)
    old_dy, old_x = SW.operands(0, 2, 2, tokens=384, out_f=24, in_f=40, dy_scale=1e-3)
    old = W.bf16_rne(W.wgrad_exact(old_dy, old_x))
    K = dy.shape[0]
    idx = np.arange(K) if order == "forward" else np.random.default_rng(5).permutation(K)
    acc = _fp32_accumulate(dy, x, idx)
    z = (W.widen_bf16(old).astype(np.float32) + acc).astype(np.float32)
    q = W.widen_bf16(W.bf16_rne(z.astype(np.float64)))
    exact = W.wgrad_accumulate_exact(old, dy, x)
    assert np.all(np.abs(q - exact) <= W.error_bound_accumulate(old, dy, x, exact))


def test_accumulate_exact_is_old_plus_product():
    dy, x = SW.small_integer_operands(8, tokens=6, out_f=4, in_f=5, vmax=2)
    old = W.bf16_rne(np.arange(20, dtype=np.float64).reshape(4, 5) - 7.0)
    got = W.wgrad_accumulate_exact(old, dy, x)
    assert np.array_equal(got, (np.arange(20).reshape(4, 5) - 7.0) + W.wgrad_exact(dy, x))


def test_accumulate_bound_is_violated_by_a_dropped_old_gradient():
    # a kernel that overwrites instead of accumulating falls outside the bound
    dy, x = SW.operands(0, 1, 3, tokens=128, out_f=16, in_f=16, dy_scale=1e-3)
    old = W.bf16_rne(W.wgrad_exact(*SW.operands(0, 3, 3, tokens=128, out_f=16, in_f=16,
                                                dy_scale=1e-3)))
    exact = W.wgrad_accumulate_exact(old, dy, x)
    q = W.widen_bf16(W.bf16_rne(W.wgrad_exact(dy, x)))
    assert np.any(np.abs(q - exact) > W.error_bound_accumulate(old, dy, x, exact))
