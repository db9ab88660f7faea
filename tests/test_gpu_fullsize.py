"""Full-size workloads in the benchmark's launch configuration.

The whole gradient set of each workload is generated on the device and run
through gnmr_step exactly as bench.py does.  At these sizes the oracle
computes a sample of units one by one: their norms (host-generated values)
and, since Alg. 1 is per unit, their GNMR, Delta-GNMR and R over the steps.
For all units the outputs are checked against properties that hold at any
size: the budget cap, candidate pool, Top_maxO order with index ties, the
lock rule and the step counters (Alg. 2; Sec. 3.3, 3.4).
"""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import streams as S
from gpu_util import controller_for, device_buffer, require_gpu
from oracle import Controller as Oracle
from synth import layout as L
from synth import recipe as R

pytestmark = pytest.mark.gpu

FULL = [("llama2-7b", 3), ("llama2-13b", 3), ("llama2-13b-layers", 3), ("moe", 4), ("fine128", 4),
        ("fine32", 4)]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def gen():
    require_gpu()
    from synth.gpu import Generator

    return Generator()


def check_properties(out, w, lock_before, alpha, beta, what):
    """Alg. 2 invariants of one step's outputs, over every unit."""
    U = w.num_units
    mask, lock, risk = out["mask"], out["lock"], out["risk"]
    g, d = out["gnmr"], out["dgnmr"]
    st = out["stats"]
    assert set(np.unique(mask)) <= {0, 1}, what
    # R = max(GNMR / alpha, Delta-GNMR / beta), the same float64 operations
    assert np.array_equal(risk, np.maximum(g / alpha, d / beta)), what
    trig = risk > 1.0
    cand = trig | (lock_before > 0)
    sel = mask.astype(bool)
    assert not np.any(sel & ~cand), f"{what}: active unit outside C_t"
    assert st["n_cand"] == int(cand.sum()) and st["n_active"] == int(sel.sum()), what
    assert st["n_trig"] == int(trig.sum()), what
    assert st["n_trig_gnmr"] == int((g / alpha > 1.0).sum()), what
    assert st["n_trig_dgnmr"] == int((d / beta > 1.0).sum()), what
    assert st["hit_maxo"] == int(cand.sum() > 0 and cand.sum() >= w.max_o), what
    if cand.sum() <= w.max_o:
        assert np.array_equal(sel, cand), f"{what}: cap not binding, A_t must equal C_t"
    else:
        assert sel.sum() == w.max_o, f"{what}: cap binding, |A_t| must be maxO"
        r_in, r_out = risk[sel], risk[cand & ~sel]
        assert r_in.min() >= r_out.max(), f"{what}: Top_maxO order"
        tie = r_in.min()
        if r_out.max() == tie:            # equal keys at the cut: smaller indices first
            assert np.flatnonzero(sel & (risk == tie)).max() < \
                np.flatnonzero(cand & ~sel & (risk == tie)).min(), what
    want = np.zeros(U, dtype=np.int32)
    want[sel & trig] = w.lock_len
    keep = sel & ~trig
    want[keep] = np.maximum(lock_before[keep] - 1, 0)
    assert np.array_equal(lock, want), f"{what}: lock rule"


@pytest.mark.parametrize("name,steps", FULL)
def test_fullsize_sampled(gen, name, steps):
    torch = require_gpu()
    w = R.get(name)
    lay = L.for_workload(w)
    U = w.num_units
    rng = np.random.default_rng(2024)
    sample = sorted({0, U - 1, int(np.argmax(w.numel)), *rng.choice(U, 3, replace=False).tolist()})
    say(f"full-size {name}: {U} units, {w.bytes_per_step / 1e9:.2f} GB/step, sample {sample}")
    buf, base, ptrs = device_buffer(torch, lay)
    ora = Oracle(len(sample), window=w.window, max_o=len(sample), lock_len=w.lock_len,
                 eps=w.eps)
    lock_before = np.zeros(U, dtype=np.int32)
    pool = ThreadPoolExecutor(max_workers=min(8, len(sample)))
    try:
        with controller_for(lay, w, ptrs) as ctl:
            # K1, K2, K3: every full-size workload is too large for the
            # single-workgroup K2 + K3 launch
            assert ctl.info()["launches_per_step"] == 3
            for t in range(1, steps + 1):
                alpha, beta = w.alpha(t), w.beta(t)
                s32 = w.scale32(t)
                gen.fill(lay, base, w.seed, t, s32)
                ctl.step(alpha, beta)
                out = ctl.query()
                hn = list(pool.map(lambda b: S.host_unit_norm(w.seed, t, b, s32[b],
                                                             w.units[b].dtype, w.units[b].numel),
                                   sample))
                ref = ora.step(hn, alpha, beta)
                for f in ("norm", "gnmr", "dgnmr", "risk"):
                    np.testing.assert_allclose(out[f][sample], getattr(ref, f), rtol=1e-5,
                                               atol=0, err_msg=f"{name} t={t} {f}")
                check_properties(out, w, lock_before, alpha, beta, f"{name} t={t}")
                lock_before = out["lock"].copy()
                say(f"  t={t} ok: stats {out['stats']}")
    finally:
        pool.shutdown()
        del buf
        torch.cuda.empty_cache()


@pytest.mark.parametrize("name,steps", [("llama2-13b", 6), ("moe", 4), ("fine32", 4),
                                        ("llama2-13b-layers", 3)])
def test_fullsize_scale_invariance(gen, name, steps):
    """GNMR is dimensionless (Sec. 3.1): with eps = 0, multiplying every value
    of unit b by 2^m_b at every step scales its norm by exactly 2^m_b (the
    squares, their fp32 and float64 sums and the square root all commute with
    a power of two away from the range limits), so GNMR, Delta-GNMR, R, the
    mask, the locks and the counters of every unit are bit-identical to the
    unscaled run, and every norm is exactly 2^m_b times the unscaled one.  A
    second context over the unscaled values gives bit-identical outputs
    (fixed work items and reduction trees, no float atomics).  At full size,
    in the benchmark's launch configuration, every unit."""
    torch = require_gpu()
    w = R.get(name)
    lay = L.for_workload(w)
    U = w.num_units
    m = np.random.default_rng(3).integers(-8, 9, size=U)
    say(f"scale invariance {name}: {U} units x {steps} steps, m in [{m.min()}, {m.max()}]")
    buf, base, ptrs = device_buffer(torch, lay)
    cfg = dict(window=w.window, max_o=w.max_o, lock_len=w.lock_len, eps=0.0)
    try:
        with controller_for(lay, ptrs=ptrs, **cfg) as plain, \
                controller_for(lay, ptrs=ptrs, **cfg) as again, \
                controller_for(lay, ptrs=ptrs, **cfg) as scaled:
            for t in range(1, steps + 1):
                s32 = w.scale32(t)
                gen.fill(lay, base, w.seed, t, s32)
                plain.step(w.alpha(t), w.beta(t))
                again.step(w.alpha(t), w.beta(t))
                a, a2 = plain.query(), again.query()
                for f in ("mask", "lock", "norm", "gnmr", "dgnmr", "risk"):
                    assert np.array_equal(a[f], a2[f]), f"{name} t={t}: {f} not repeatable"
                gen.fill(lay, base, w.seed, t, (s32 * np.exp2(m)).astype(np.float32))
                scaled.step(w.alpha(t), w.beta(t))
                b = scaled.query()
                what = f"{name} t={t}"
                for f in ("mask", "lock", "gnmr", "dgnmr", "risk"):
                    assert np.array_equal(a[f], b[f]), f"{what}: {f} differs"
                assert a["stats"] == b["stats"], what
                assert np.array_equal(b["norm"], a["norm"] * np.exp2(m)), f"{what}: norm"
    finally:
        del buf
        torch.cuda.empty_cache()
