"""Pins of the actuator oracle (per-token fake quantisation, App. E.2)
against the floating-point format definitions and brute force.  CPU only."""
import itertools

import numpy as np
import pytest

from oracle import fakequant as FQ

# (exponent bits, mantissa bits, bias, has the all-ones-exponent values as finite)
DEFS = {1: (2, 1, 1, True), 2: (3, 2, 3, True), 3: (4, 3, 7, "e4m3"), 4: (5, 2, 15, False)}


def grid(fmt):
    """Every non-negative representable value, from the bit-field definition."""
    eb, mb, bias, allones = DEFS[fmt]
    vals = set()
    for E, M in itertools.product(range(2 ** eb), range(2 ** mb)):
        if E == 2 ** eb - 1:
            if allones is False:                    # E5M2: inf / NaN
                continue
            if allones == "e4m3" and M == 2 ** mb - 1:   # E4M3: only S.1111.111 is NaN
                continue
        if E == 0:
            v = (M / 2 ** mb) * 2.0 ** (1 - bias)   # subnormal
        else:
            v = (1 + M / 2 ** mb) * 2.0 ** (E - bias)
        vals.add(v)
    return np.array(sorted(vals))


def test_known_grids():
    assert grid(1).tolist() == [0, 0.5, 1, 1.5, 2, 3, 4, 6]
    assert grid(2).max() == 28 and grid(3).max() == 448 and grid(4).max() == 57344
    assert grid(3).min() == 0 and sorted(grid(3))[1] == 2.0 ** -9


@pytest.mark.parametrize("fmt", [1, 2, 3, 4])
def test_round_to_format_is_nearest_grid_value(fmt):
    g = grid(fmt)
    rng = np.random.default_rng(fmt)
    fmax = g.max()
    y = np.concatenate([
        rng.uniform(-1.2 * fmax, 1.2 * fmax, 20000),
        rng.uniform(-4 * g[1], 4 * g[1], 5000),                 # subnormal range
        np.concatenate([g, -g, (g[1:] + g[:-1]) / 2]),          # grid points and exact ties
    ]).astype(np.float32)
    got = FQ.round_to_format(y, fmt)
    a = np.abs(y).astype(np.float64)
    idx = np.searchsorted(g, a)
    lo = g[np.clip(idx - 1, 0, len(g) - 1)]
    hi = g[np.clip(idx, 0, len(g) - 1)]
    dlo, dhi = a - lo, hi - a
    # ties go to the value whose significand is even: position in the binade grid
    eb, mb, bias, _ = DEFS[fmt]
    def even(v):
        if v == 0:
            return True
        e = max(np.floor(np.log2(v)), 1 - bias)
        return int(round(v / 2.0 ** (e - mb))) % 2 == 0
    want = np.where(dlo < dhi, lo, hi)
    tie = dlo == dhi
    want[tie] = [l if even(l) else h for l, h in zip(lo[tie], hi[tie])]
    want = np.copysign(np.minimum(want, g.max()), y)
    assert np.array_equal(got.astype(np.float64), want)
    assert np.array_equal(np.signbit(got), np.signbit(y))


@pytest.mark.parametrize("fmt", [1, 2, 3, 4])
def test_fakequant_rows_properties(fmt):
    rng = np.random.default_rng(10 + fmt)
    x = rng.normal(size=(33, 200)).astype(np.float32) * 10.0 ** rng.uniform(-6, 2, (33, 1))
    x[3] = 0.0
    x[5, 7] = 500.0                                             # an outlier token
    xb = FQ.f32_to_bf16(x)
    out = FQ.fakequant_rows(xb, fmt)
    xf, of = FQ.bf16_to_f32(xb), FQ.bf16_to_f32(out)
    assert np.all(of[3] == 0)
    g = grid(fmt)
    amax = np.abs(xf).max(axis=1)
    for r in range(x.shape[0]):
        if amax[r] == 0:
            continue
        s = np.float32(amax[r] / np.float32(g.max()))
        inv = np.float32(np.float32(g.max()) / amax[r])
        y = np.abs((xf[r] * inv).astype(np.float32)).astype(np.float64)
        # the output is the scaled-back nearer of the two representable values
        # around |y| (either one at an exact tie), rounded to bf16
        i = np.clip(np.searchsorted(g, y), 1, len(g) - 1)
        lo, hi = g[i - 1], g[i]
        lo = np.where(y > g.max(), g.max(), lo)
        hi = np.where(y > g.max(), g.max(), hi)
        blo = FQ.bf16_to_f32(FQ.f32_to_bf16((lo * s).astype(np.float32)))
        bhi = FQ.bf16_to_f32(FQ.f32_to_bf16((hi * s).astype(np.float32)))
        o = np.abs(of[r])
        assert np.all(np.where(y - lo < hi - y, o == blo, np.where(y - lo > hi - y, o == bhi,
                                                                     (o == blo) | (o == bhi))))
        # the largest element maps back to about amax
        assert abs(np.abs(of[r]).max() - amax[r]) <= 1e-2 * amax[r]
    # powers of two commute with the quantiser
    out2 = FQ.fakequant_rows(FQ.f32_to_bf16(xf * np.float32(2.0 ** 5)), fmt)
    assert np.array_equal(FQ.bf16_to_f32(out2), of * np.float32(2.0 ** 5))


def test_int8_round_is_nearest_integer():
    """INT8: brute force over the 255-value grid, ties to the even integer,
    saturation at +-127, signs (and -0) kept."""
    g = np.arange(0, 128, dtype=np.float64)
    rng = np.random.default_rng(55)
    y = np.concatenate([rng.uniform(-140, 140, 20000), rng.uniform(-2, 2, 2000),
                        np.concatenate([g, -g, g[:-1] + 0.5, -(g[:-1] + 0.5)]),
                        [127.49, 127.5, 127.51, 128.0, 1e6, -1e6, 0.0, -0.0, 1e-40]]
                       ).astype(np.float32)
    got = FQ.round_to_int(y, 5).astype(np.float64)
    a = np.abs(y).astype(np.float64)
    d = np.abs(a[:, None] - g[None, :])
    best = d.min(axis=1)
    cand = d == best[:, None]
    # among equidistant grid values take the even one (an integer tie)
    pick = np.where(cand.sum(axis=1) > 1, np.argmax(cand & (g[None, :] % 2 == 0), axis=1),
                    np.argmax(cand, axis=1))
    want = np.copysign(g[pick], y)
    assert np.array_equal(got, want)
    assert np.array_equal(np.signbit(got), np.signbit(y))
    assert FQ.round_to_int(np.float32([2.5, 3.5, -2.5, 126.5]), 5).tolist() == [2, 4, -2, 126]


def test_int8_rows():
    """INT8 per-token rows: every output is an integer multiple of amax/127
    (up to the final bf16 rounding), the largest element returns to amax, and
    the quantisation error of each element is at most half a step."""
    rng = np.random.default_rng(56)
    x = rng.normal(size=(17, 300)).astype(np.float32) * 10.0 ** rng.uniform(-5, 3, (17, 1))
    x[4] = 0.0
    x[4, ::3] = -0.0                                           # an all-zero token with -0s
    x[6, 9] = -800.0
    xb = FQ.f32_to_bf16(x)
    out = FQ.fakequant_rows(xb, 5)
    xf, of = FQ.bf16_to_f32(xb).astype(np.float64), FQ.bf16_to_f32(out).astype(np.float64)
    assert np.all(of[4] == 0) and not np.any(np.signbit(of[4]))
    for r in range(x.shape[0]):
        amax = np.abs(xf[r]).max()
        if amax == 0:
            continue
        s = amax / 127.0
        k = np.rint(of[r] / s)
        assert np.all(np.abs(k) <= 127)
        # bf16 keeps 8 significant bits: within 2^-8 of k s (plus fp32 slack)
        assert np.all(np.abs(of[r] - k * s) <= 2.0 ** -8 * np.abs(k * s) + 1e-6 * s)
        assert np.all(np.abs(xf[r] - k * s) <= 0.5 * s * (1 + 1e-5))
        assert abs(np.abs(of[r]).max() - amax) <= 2.0 ** -8 * amax
        assert np.array_equal(np.signbit(of[r]), np.signbit(xf[r]))
    # the integer grid: INT8 of data already on a grid of amax/127 is exact
    grid_rows = (np.arange(-127, 128, dtype=np.float32) * np.float32(2.0 ** -3))[None, :]
    exact = FQ.fakequant_rows(FQ.f32_to_bf16(grid_rows), 5)
    assert np.array_equal(FQ.bf16_to_f32(exact), grid_rows)


def test_f32_to_bf16_is_nearest_even():
    """fp32 -> bf16 against the two neighbouring bf16 values in float64:
    the nearer one, the one with the even last bit at an exact tie."""
    rng = np.random.default_rng(57)
    u = rng.integers(0, 0x7F7F0000, 50000, dtype=np.uint32)
    u[:64] = (rng.integers(0x00800000, 0x7F000000, 64, dtype=np.uint32) & 0xFFFF0000) | 0x8000
    u = np.concatenate([u, u | np.uint32(0x80000000)])      # both signs
    x = u.view(np.float32)
    got = FQ.f32_to_bf16(x)
    lo = (u & np.uint32(0xFFFF0000))
    hi = lo + np.uint32(0x10000)
    xl, xh = lo.view(np.float32).astype(np.float64), hi.view(np.float32).astype(np.float64)
    d_lo = np.abs(x.astype(np.float64) - xl)
    d_hi = np.abs(x.astype(np.float64) - xh)
    lo16, hi16 = (lo >> 16).astype(np.uint16), (hi >> 16).astype(np.uint16)
    want = np.where(d_lo < d_hi, lo16, np.where(d_hi < d_lo, hi16,
                                                 np.where(lo16 % 2 == 0, lo16, hi16)))
    assert np.array_equal(got, want)
    assert FQ.f32_to_bf16(np.float32([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8])).tolist() == \
        [0x3F80, 0x3F82]


def test_identity_format_and_actuate():
    rng = np.random.default_rng(3)
    a = FQ.f32_to_bf16(rng.normal(size=(4, 16)).astype(np.float32))
    b = FQ.f32_to_bf16(rng.normal(size=(2, 8)).astype(np.float32))
    out = FQ.actuate([a, b], [1, 0], fmt_lo=1, fmt_hi=0)
    assert np.array_equal(out[0], a)                         # recovery path: BF16 untouched
    assert np.array_equal(out[1], FQ.fakequant_rows(b, 1))    # low-cost path: E2M1
