"""Non-finite and out-of-range gradient elements through the whole step
(K1 -> K2 -> K3, gnmr_step) against the oracle.

Non-finite norms are outside the paper; the reading both sides follow: a
unit whose gradient holds a NaN gets n = NaN, one with an Inf (and no NaN)
n = +inf, and one whose sum of squares reaches 2^128 (the end of the fp32
range the gradient pass accumulates in) n = +inf.  Such a unit gets GNMR =
Delta-GNMR = R = +inf, keeps its historical mean A, pushes 1.0 into its
queue Q and counts in n_nonfinite; +inf risks rank first, ties by index.

The special values sit inside an item body, in a misaligned head, in a
misaligned tail, as fp32 squares that overflow, and as item partials that
are finite while the unit's total is not.  Steps without special values
follow, so the kept A and Q are checked through the later GNMR and
Delta-GNMR.  Bars: masks, locks and counters bit-exact; finite norms and
ratios within 1e-5; non-finite values of the same kind (NaN or +inf).
"""
import sys

import numpy as np
import pytest

from gpu_util import controller_for, device_buffer, require_gpu
from oracle import Controller as Oracle
from oracle import unit_norm as oracle_norm
from synth import layout as L
from synth import values as V

pytestmark = pytest.mark.gpu

BF16, F32 = V.DTYPE_BF16, V.DTYPE_F32
SEED = 21


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


# unit: (dtype, pieces, shift in bytes of each piece)
UNITS = [
    (BF16, [100_003], [0]),            # 0: NaN inside an item body
    (F32, [50_001], [4]),              # 1: +Inf in the misaligned head
    (BF16, [35_000, 35_001], [2, 6]),  # 2: -Inf in the misaligned tail, later NaN
    (F32, [20_000], [0]),              # 3: squares of 2^64 overflow fp32
    (BF16, [40_000], [0]),             # 4: 2^62 elements: finite, near the top of the range
    (BF16, [80_000], [0]),             # 5: item partials finite, unit total >= 2^128
    (BF16, [65_536], [0]),
    (F32, [33_333], [8]),
    (BF16, [1], [2]),                  # 8, 9: monitored only (their norms are a
    (F32, [7], [12]),                  #   handful of values, so their ratios roam)
]
RECOVERABLE = np.array([1] * 8 + [0, 0], np.uint8)

NINF_BF16 = int(V.f32_to_bf16_bits(np.array([-np.inf], np.float32))[0])
NAN_BF16 = 0x7FC0


def bf16_bits(v):
    return int(V.f32_to_bf16_bits(np.array([v], np.float32))[0])


# step -> [(unit, element of the unit, value as bits of its dtype)]
PLANTS = {
    2: [(0, 40_000, NAN_BF16),
        (1, 0, int(np.array([np.inf], np.float32).view(np.uint32)[0])),
        (2, 70_000, NINF_BF16),
        (3, 5, int(np.array([2.0 ** 64], np.float32).view(np.uint32)[0])),
        (3, 6, int(np.array([-(2.0 ** 64)], np.float32).view(np.uint32)[0])),
        (4, 10, bf16_bits(2.0 ** 62)), (4, 20_000, bf16_bits(-(2.0 ** 62))),
        (4, 39_999, bf16_bits(2.0 ** 62)), (4, 30_000, bf16_bits(2.0 ** 62))],
    4: [(2, 35_000, NAN_BF16),
        # two 2^63 in item 0 and three in item 1: partials 2^127 and 1.5 * 2^127
        (5, 3, bf16_bits(2.0 ** 63)), (5, 30_000, bf16_bits(-(2.0 ** 63))),
        (5, 40_000, bf16_bits(2.0 ** 63)), (5, 50_000, bf16_bits(2.0 ** 63)),
        (5, 65_000, bf16_bits(-(2.0 ** 63)))],
}
STEPS = 6


def layout():
    sizes = [sum(p) for _, p, _ in UNITS]
    dtypes = [d for d, _, _ in UNITS]
    pieces = [p for _, p, _ in UNITS]
    shift = [s for _, _, sh in UNITS for s in sh]
    return L.build(sizes, dtypes, pieces=pieces, shift=shift)


def host_unit(lay, t, b, scale, plants):
    """Unit b's segments at step t as (values, dtype), plants applied."""
    dtype = UNITS[b][0]
    full = V.unit_values(SEED, t, b, float(scale[b]), dtype, 0, sum(UNITS[b][1]))
    full = full.copy()
    for u, e, bits in plants:
        if u == b:
            full[e] = bits if dtype == BF16 else np.array([bits], np.uint32).view(np.float32)[0]
    segs, start = [], 0
    for n in UNITS[b][1]:
        segs.append((full[start:start + n], dtype))
        start += n
    return segs


def plant_on_device(torch, buf, lay, plants):
    for b, e, bits in plants:
        s = int(lay.unit_seg_off[b])
        while e >= int(lay.seg_unit_base[s]) + int(lay.seg_numel[s]):
            s += 1
        esz = V.DTYPE_SIZE[UNITS[b][0]]
        off = int(lay.seg_byte_off[s]) + (e - int(lay.seg_unit_base[s])) * esz
        raw = np.array([bits], np.uint16 if esz == 2 else np.uint32).view(np.uint8)
        buf[off:off + esz] = torch.from_numpy(raw.copy()).to(buf.device)


def assert_guarded(ref, alpha, beta, window, t, max_o):
    """The decisions of this fixed-seed stream are far from every threshold
    (so that fp32 sums give the same masks as float64 ones)."""
    rec = RECOVERABLE.astype(bool) & np.isfinite(ref.norm)
    assert np.all(np.abs(ref.gnmr[rec] / alpha - 1) > 1e-4), t
    if t > window:
        assert np.all(np.abs(ref.dgnmr[rec] / beta - 1) > 1e-4), t
    pool = np.sort(ref.risk[RECOVERABLE.astype(bool) & ((ref.risk > 1) | (ref.lock > 0) |
                                                        (ref.mask > 0))])[::-1]
    if pool.size > max_o > 0:
        a, b = pool[max_o - 1], pool[max_o]
        assert a == b or (a - b) / a > 1e-4, (t, a, b)


@pytest.mark.parametrize("max_o", [8, 2])
def test_nonfinite_and_out_of_range_elements_through_k1(max_o):
    torch = require_gpu()
    from synth.gpu import Generator

    gen = Generator()
    lay = layout()
    U = lay.num_units
    say("non-finite elements through gnmr_step: units", U, "segments", lay.num_segments,
        "max_o", max_o)
    buf, base, ptrs = device_buffer(torch, lay)
    scale = np.full(U, 1e-3, np.float32)
    cfg = dict(window=3, max_o=max_o, lock_len=2, eps=1e-12)
    ora = Oracle(U, recoverable=RECOVERABLE, **cfg)
    seen_kinds = set()
    with controller_for(lay, ptrs=ptrs, recoverable=RECOVERABLE, **cfg) as ctl:
        for t in range(1, STEPS + 1):
            plants = PLANTS.get(t, [])
            gen.fill(lay, base, SEED, t, scale)
            plant_on_device(torch, buf, lay, plants)
            torch.cuda.synchronize()
            ctl.step(1.5, 1.5)
            out = ctl.query()
            norms = np.array([oracle_norm(host_unit(lay, t, b, scale, plants)) for b in range(U)])
            ref = ora.step(norms, 1.5, 1.5)
            assert_guarded(ref, 1.5, 1.5, cfg["window"], t, max_o)
            what = f"t={t} max_o={max_o}"
            assert np.array_equal(out["mask"], ref.mask), (what, out["mask"], ref.mask)
            assert np.array_equal(out["lock"], ref.lock), (what, out["lock"], ref.lock)
            for k, v in ref.stats.items():
                assert out["stats"][k] == v, (what, k, out["stats"][k], v)
            fin = np.isfinite(ref.norm)
            for b in np.flatnonzero(~fin):
                kind = "nan" if np.isnan(ref.norm[b]) else "inf"
                seen_kinds.add((b, kind))
                assert (np.isnan(out["norm"][b]) if kind == "nan"
                        else out["norm"][b] == np.inf), (what, b, out["norm"][b], ref.norm[b])
                for f in ("gnmr", "dgnmr", "risk"):
                    assert out[f][b] == np.inf and getattr(ref, f)[b] == np.inf, (what, b, f)
            for f in ("norm", "gnmr", "dgnmr", "risk"):
                np.testing.assert_allclose(out[f][fin], getattr(ref, f)[fin], rtol=1e-5, atol=0,
                                           err_msg=f"{what} {f}")
    # every planted kind showed up as intended
    assert seen_kinds == {(0, "nan"), (1, "inf"), (2, "inf"), (3, "inf"), (2, "nan"),
                          (5, "inf")}, seen_kinds
