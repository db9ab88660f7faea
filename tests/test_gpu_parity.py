"""Parity of the HIP controller pass (through the C ABI) with the CPU oracle.

Bars: masks, locks and counters bit-exact; norms, GNMR, Delta-GNMR and R
within 1e-5 relative (fp32 accumulation of squares against float64).  Inputs
are seeded and synthetic; decisions are kept at least 1e-4 away from every
threshold (see tests/streams.py) so that bit-exact masks are well defined.
"""
import sys

import numpy as np
import pytest

import streams as S
from gpu_util import assert_step_matches, controller_for, device_buffer, require_gpu
from oracle import Controller as Oracle
from oracle import sumsq as oracle_sumsq
from oracle import unit_norm as oracle_norm
from synth import layout as L
from synth import recipe as R
from synth import values as V

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def gen():
    require_gpu()
    from synth.gpu import Generator

    return Generator()


def test_tiny_end_to_end(gen):
    torch = require_gpu()
    w = R.get("tiny")
    say("tiny end-to-end:", w.description)
    nudge, _, ref, alphas, betas = S.guarded_stream(
        w, lambda t, s32, units: S.host_norms(w, t, s32, units))
    lay = L.for_workload(w)
    buf, base, ptrs = device_buffer(torch, lay)
    with controller_for(lay, w, ptrs) as ctl:
        # K1, then K2 + K3 in one workgroup (28 units of a few items each)
        assert ctl.info()["launches_per_step"] == 2
        for t in range(1, w.steps + 1):
            gen.fill(lay, base, w.seed, t, w.scale32(t, nudge[t - 1]))
            ctl.step(alphas[t - 1], betas[t - 1])
            assert_step_matches(ctl.query(), ref[t - 1], what=f"t={t}")
    # the generator is bit-identical to the host twin (last step, two units)
    for b in (0, 27):
        s = int(lay.seg_byte_off[b])
        n = int(lay.seg_numel[b])
        dev = buf[s:s + 4 * n].cpu().numpy().view(np.float32)
        host = V.unit_values(w.seed, w.steps, b, float(w.scale32(w.steps, nudge[-1])[b]),
                             V.DTYPE_F32, 0, n)
        assert np.array_equal(dev, host)


def ragged_layout(rng, misaligned: bool):
    sizes = [0, 1, 7, 8, 9, 4095, 32767, 32768, 32769, 65536 * 3 + 5, 1_000_003, 123_457, 2]
    dtypes = [int(rng.integers(0, 2)) for _ in sizes]
    pieces = []
    for n in sizes:
        if n > 20 and rng.random() < 0.6:
            cuts = sorted(rng.choice(np.arange(1, n), size=int(rng.integers(1, 4)), replace=False))
            p = np.diff([0, *cuts, n]).tolist()
            p.insert(int(rng.integers(0, len(p) + 1)), 0)     # an empty segment
            pieces.append(p)
        elif n == 0:
            pieces.append([])                                # a unit with no segment
        else:
            pieces.append([n])
    nseg = sum(len(p) for p in pieces)
    shift = None
    if misaligned:
        shift = []
        for b, p in enumerate(pieces):
            esz = V.DTYPE_SIZE[dtypes[b]]
            shift += [int(rng.integers(0, 16 // esz)) * esz for _ in p]
        assert len(shift) == nseg
    return L.build(sizes, dtypes, pieces=pieces, shift=shift), sizes, dtypes, pieces


@pytest.mark.parametrize("misaligned", [False, True])
def test_sumsq_ragged_layouts(gen, misaligned):
    torch = require_gpu()
    rng = np.random.default_rng(7 if misaligned else 8)
    lay, sizes, dtypes, pieces = ragged_layout(rng, misaligned)
    say("ragged sumsq: misaligned", misaligned, "segments", lay.num_segments)
    buf, base, ptrs = device_buffer(torch, lay)
    scale = (10.0 ** rng.uniform(-4, -2, size=len(sizes))).astype(np.float32)
    gen.fill(lay, base, 5, 3, scale)
    out = torch.zeros(len(sizes), dtype=torch.float64, device="cuda")
    out2 = torch.zeros_like(out)
    with controller_for(lay, ptrs=ptrs, window=5, max_o=2, lock_len=1, eps=0.0) as ctl:
        ctl.sumsq(out)
        ctl.sumsq(out2)
        torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.array_equal(got, out2.cpu().numpy())                 # deterministic
    for b, n in enumerate(sizes):
        segs, start = [], 0
        for m in pieces[b]:
            segs.append((V.unit_values(5, 3, b, float(scale[b]), dtypes[b], start, m), dtypes[b]))
            start += m
        ref = oracle_sumsq(segs)
        if n == 0:
            assert got[b] == 0.0
        else:
            assert abs(got[b] - ref) <= 5e-6 * ref, (b, n, got[b], ref)


@pytest.mark.parametrize("case", ["ragged_misaligned", "bf16_128_units", "bf16_1024_units"])
def test_small_step_matches_norm_path(gen, case):
    """A small workload's step (K1, then K2 and K3 in one workgroup) against
    the same steps taken as K1 and the unit sums, then the controller from
    those norms: every output bit-identical, step after step; the norms also
    within the bar of the oracle's sum of squares.  bf16_1024_units sits at
    the single workgroup's limit: 1,024 units of one work item each."""
    torch = require_gpu()
    rng = np.random.default_rng(11)
    if case == "ragged_misaligned":
        lay, sizes, dtypes, pieces = ragged_layout(rng, True)
    elif case == "bf16_128_units":
        sizes = [524289] + [524288] * 127                # 1 MiB of bf16 each, one ragged
        dtypes = [V.DTYPE_BF16] * 128
        pieces = [[n] for n in sizes]
        lay = L.build(sizes, dtypes)
    else:
        sizes = [20001] + [20000] * 1023                 # 40 kB of bf16 each, one ragged
        dtypes = [V.DTYPE_BF16] * 1024
        pieces = [[n] for n in sizes]
        lay = L.build(sizes, dtypes)
    launches = 2
    U = len(sizes)
    say("small step vs norm path:", case, "units", U, "segments", lay.num_segments)
    buf, base, ptrs = device_buffer(torch, lay)
    cfg = dict(window=3, max_o=3, lock_len=2, eps=1e-12)
    ss = torch.zeros(U, dtype=torch.float64, device="cuda")
    with controller_for(lay, ptrs=ptrs, **cfg) as one, \
            controller_for(lay, ptrs=ptrs, **cfg) as ref:
        assert one.info()["launches_per_step"] == launches
        scale = (10.0 ** rng.uniform(-4, -2, size=U)).astype(np.float32)
        for t in range(1, 7):
            step_scale = scale.copy()
            step_scale[rng.choice(U, size=min(3, U), replace=False)] *= 20.0   # spikes
            gen.fill(lay, base, 9, t, step_scale)
            one.step(1.5, 1.3)
            ref.sumsq(ss)
            ref.step_from_norms(torch.sqrt(ss), 1.5, 1.3)
            a, b = one.query(), ref.query()
            for k in ("mask", "lock", "norm", "gnmr", "dgnmr", "risk"):
                assert np.array_equal(a[k], b[k]), (case, t, k)
            assert a["stats"] == b["stats"], (case, t)
            assert a["stats"]["t"] == t
            for u in (range(U) if U <= 128 else sorted({0, 1, U - 1, *range(0, U, 37)})):
                segs, start = [], 0
                for m in pieces[u]:
                    segs.append((V.unit_values(9, t, u, float(step_scale[u]), dtypes[u], start, m),
                                 dtypes[u]))
                    start += m
                want = np.sqrt(oracle_sumsq(segs))
                assert abs(a["norm"][u] - want) <= 1e-5 * want, (case, t, u, a["norm"][u], want)


@pytest.mark.parametrize("name", ["tiny", "llama2-7b", "llama2-13b", "moe", "fine128", "fine32"])
def test_logic_from_norms(name):
    """Alg. 1 + Alg. 2 on norm streams shaped like each workload: with identical
    float64 norms both sides do identical IEEE arithmetic."""
    torch = require_gpu()
    w = R.get(name)
    norms = R.surrogate_norms(w)
    say("norm-level parity:", name, "units", w.num_units, "steps", w.steps)
    from paper_2606_00539_amd import Controller

    ora = Oracle(w.num_units, window=w.window, max_o=w.max_o, lock_len=w.lock_len, eps=w.eps)
    dn = torch.empty(w.num_units, dtype=torch.float64, device="cuda")
    with Controller(w.num_units, w.window, w.max_o, w.lock_len, w.eps, np.zeros(w.num_units + 1),
                    [], []) as ctl:
        for t in range(1, w.steps + 1):
            dn.copy_(torch.from_numpy(norms[t - 1]))
            ctl.step_from_norms(dn, w.alpha(t), w.beta(t))
            ref = ora.step(norms[t - 1], w.alpha(t), w.beta(t))
            assert_step_matches(ctl.query(), ref, rtol=1e-14, what=f"{name} t={t}")


def upload_units(torch, arrays):
    """Place host arrays (float32) as one fp32 segment each; returns the layout
    and the buffer."""
    lay = L.build([a.size for a in arrays], [V.DTYPE_F32] * len(arrays))
    buf, base, ptrs = device_buffer(torch, lay)
    for a, off in zip(arrays, lay.seg_byte_off):
        buf[int(off):int(off) + 4 * a.size].copy_(torch.from_numpy(a.view(np.uint8)))
    return lay, buf, ptrs


def test_constant_magnitude_is_exactly_one():
    torch = require_gpu()
    rng = np.random.default_rng(0)
    mags = [2.0 ** -10, 2.0 ** -7]
    lay = None
    with torch.no_grad():
        arrays = [np.where(rng.random(40_000 + 17 * i) < 0.5, -m, m).astype(np.float32)
                  for i, m in enumerate(mags)]
        lay, buf, ptrs = upload_units(torch, arrays)
        with controller_for(lay, ptrs=ptrs, window=5, max_o=1, lock_len=2, eps=0.0) as ctl:
            for t in range(1, 21):
                for a, off in zip(arrays, lay.seg_byte_off):     # fresh signs, same magnitude
                    rng.shuffle(a)
                    buf[int(off):int(off) + 4 * a.size].copy_(torch.from_numpy(a.view(np.uint8)))
                ctl.step(1.1, 1.5)
                out = ctl.query()
                assert np.all(out["gnmr"] == 1.0) and np.all(out["dgnmr"] == 1.0)
                assert out["mask"].sum() == 0


def test_spike_closed_form_on_gpu():
    torch = require_gpu()
    c, N, t0, k, delta = 2.0 ** -10, 1 << 16, 9, 20, 5
    base = np.full(N, c, dtype=np.float32)
    base[1::2] *= -1
    lay, buf, ptrs = upload_units(torch, [base.copy(), base.copy()])
    off = int(lay.seg_byte_off[0])
    with controller_for(lay, ptrs=ptrs, window=delta, max_o=1, lock_len=3, eps=0.0) as ctl:
        hist = []
        for t in range(1, t0 + 4):
            g = base * np.float32(k if t == t0 else 1)
            buf[off:off + 4 * N].copy_(torch.from_numpy(g.view(np.uint8)))
            ctl.step(1.1, 1.5)
            out = ctl.query()
            hist.append(out)
        assert hist[t0 - 1]["gnmr"][0] == k and hist[t0 - 1]["dgnmr"][0] == k
        assert hist[t0 - 1]["mask"].tolist() == [1, 0]
        assert abs(hist[t0]["gnmr"][0] - t0 / (t0 - 1 + k)) < 1e-15
        assert abs(hist[t0]["dgnmr"][0] - delta * t0 / ((t0 - 1 + k) * (delta - 1 + k))) < 1e-15
        assert [h["mask"][0] for h in hist[t0 - 1:]] == [1, 1, 1, 1]   # lock 3 holds


def test_state_roundtrip_is_bitwise():
    torch = require_gpu()
    from paper_2606_00539_amd import Controller

    w = R.get("moe")
    norms = R.surrogate_norms(w)
    dn = torch.empty(w.num_units, dtype=torch.float64, device="cuda")
    mk = lambda: Controller(w.num_units, w.window, w.max_o, w.lock_len, w.eps,
                            np.zeros(w.num_units + 1), [], [])
    a, b = mk(), mk()
    for t in range(1, 13):
        dn.copy_(torch.from_numpy(norms[t - 1]))
        a.step_from_norms(dn, w.alpha(t), w.beta(t))
    b.set_state(a.get_state())
    for t in range(13, w.steps + 1):
        dn.copy_(torch.from_numpy(norms[t - 1]))
        a.step_from_norms(dn, w.alpha(t), w.beta(t))
        b.step_from_norms(dn, w.alpha(t), w.beta(t))
        qa, qb = a.query(), b.query()
        for f in ("mask", "lock", "norm", "gnmr", "dgnmr", "risk"):
            assert np.array_equal(qa[f], qb[f])
        assert qa["stats"] == qb["stats"]
    a.close()
    b.close()


@pytest.mark.parametrize("case", ["maxo0", "alpha_below_one", "nonfinite", "not_recoverable",
                                  "window1_lock0"])
def test_edge_cases(case):
    torch = require_gpu()
    from paper_2606_00539_amd import Controller

    rng = np.random.default_rng(3)
    U, T = 300, 24
    norms = np.exp(rng.normal(scale=0.3, size=(T, U)))
    norms[10, 5] *= 30
    window, max_o, lock_len, alpha = 5, 8, 3, 1.1
    rec = None
    if case == "maxo0":
        max_o = 0
    elif case == "alpha_below_one":
        alpha = 0.4
    elif case == "nonfinite":
        norms[12, 7] = np.nan
        norms[12, 9] = np.inf
        norms[13, 7] = np.inf
    elif case == "not_recoverable":
        rec = (rng.random(U) < 0.5).astype(np.uint8)
        rec[5] = 0
    elif case == "window1_lock0":
        window, lock_len = 1, 0
    ora = Oracle(U, window=window, max_o=max_o, lock_len=lock_len, eps=1e-12, recoverable=rec)
    dn = torch.empty(U, dtype=torch.float64, device="cuda")
    with Controller(U, window, max_o, lock_len, 1e-12, np.zeros(U + 1), [], [],
                    recoverable=rec) as ctl:
        for t in range(1, T + 1):
            dn.copy_(torch.from_numpy(norms[t - 1]))
            ctl.step_from_norms(dn, alpha, 1.5)
            ref = ora.step(norms[t - 1], alpha, 1.5)
            assert_step_matches(ctl.query(), ref, rtol=1e-14, what=f"{case} t={t}")


def test_abi_errors_leave_state_unchanged():
    torch = require_gpu()
    from paper_2606_00539_amd import Controller, GnmrError
    from paper_2606_00539_amd import binding as B

    U = 4
    dn = torch.ones(U, dtype=torch.float64, device="cuda")
    with Controller(U, 5, 1, 1, 0.0, np.zeros(U + 1), [], []) as ctl:
        with pytest.raises(GnmrError) as e:
            ctl.query()
        assert e.value.status == B.GNMR_E_STATE
        ctl.step_from_norms(dn, 1.1, 1.5)
        blob = ctl.get_state()
        for a, b_ in ((0.0, 1.5), (1.1, -1.0), (float("inf"), 1.5), (1.1, float("nan"))):
            with pytest.raises(GnmrError) as e:
                ctl.step_from_norms(dn, a, b_)
            assert e.value.status == B.GNMR_E_INVALID
        assert ctl.get_state() == blob
        assert ctl.query()["stats"]["t"] == 1
        with pytest.raises(GnmrError):
            ctl.set_state(blob[:-1])
    # a misaligned segment pointer is rejected
    buf = torch.zeros(1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(GnmrError) as e:
        Controller(1, 5, 1, 1, 0.0, [0, 1], [10], [B.GNMR_F32], [buf.data_ptr() + 2])
    assert e.value.status == B.GNMR_E_INVALID
    # no pointers bound and none passed
    with Controller(1, 5, 1, 1, 0.0, [0, 1], [10], [B.GNMR_F32]) as ctl:
        with pytest.raises(GnmrError) as e:
            ctl.step(1.1, 1.5)
        assert e.value.status == B.GNMR_E_INVALID
        ctl.step(1.1, 1.5, seg_ptr=[buf.data_ptr()])
        ctl.step(1.1, 1.5)                                   # reuses bound pointers
        assert ctl.query()["stats"]["t"] == 2


@pytest.mark.parametrize("case", ["small_pool_ties_at_cut", "pool_at_count_limit",
                                  "pool_over_count_limit", "small_tie_in_radix", "few_ties_at_cut",
                                  "mid_pool_ties_at_cut", "many_ties_at_cut", "pool_at_capacity",
                                  "huge_pool"])
def test_selection_paths(case):
    """Top_maxO through each selection path of the kernel: small pools (up
    to 128 candidates) ranked by direct counting, with index-ordered ties at
    the cut and at the size limit; larger pools by radix select in LDS, with
    the early finish on a small bucket holding a tie at the cut
    (small_tie_in_radix), with larger ties at the cut sorted
    (few_ties_at_cut, mid_pool_ties_at_cut), with more ties than the tie
    buffer, and right at the LDS pool's capacity (12,288); more candidates
    than that over the global keys."""
    torch = require_gpu()
    from paper_2606_00539_amd import Controller

    rng = np.random.default_rng(11)
    U, T, max_o, alpha = 3000, 12, 64, 1.1
    base = np.exp(rng.normal(scale=0.05, size=(T, U)))
    if case == "small_pool_ties_at_cut":
        # 100 candidates: 20 distinct spikes, a 60-unit tie holding the cut,
        # 20 weaker spikes below it
        perm = rng.permutation(U)
        base = np.exp(rng.normal(scale=0.01, size=(T, U)))   # no natural triggers
        tied, strong, weak = perm[:60], perm[60:80], perm[80:100]
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
        base[9, strong] *= 18.0 + np.arange(20)
        base[9, weak] *= 2.0
    elif case in ("pool_at_count_limit", "pool_over_count_limit"):
        n = 128 if case == "pool_at_count_limit" else 129
        base = np.exp(rng.normal(scale=0.01, size=(T, U)))   # no natural triggers
        base[9, rng.permutation(U)[:n]] *= 6.0 + rng.random(n)
    elif case == "small_tie_in_radix":
        # 400 candidates: 40 distinct spikes, a 60-unit tie holding the cut (the
        # radix select finishes early on a bucket of at most 64), 300 weaker
        perm = rng.permutation(U)
        base = np.exp(rng.normal(scale=0.01, size=(T, U)))   # no natural triggers
        tied, strong, weak = perm[:60], perm[60:100], perm[100:400]
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
        base[9, strong] *= 18.0 + np.arange(40)
        base[9, weak] *= 2.0 + 0.01 * rng.random(300)
    elif case == "few_ties_at_cut":
        # 300 units share one norm stream and spike together; 20 spike harder
        tied = rng.choice(U, 300, replace=False)
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
        base[9, tied[:20]] *= 3.0
        base[9, tied[:20]] += np.arange(20)       # distinct keys above the tie
    elif case == "mid_pool_ties_at_cut":
        # about 2,000 candidates: 20 distinct spikes, a 300-unit tie holding
        # the cut, and 1,700 weaker spikes below it
        perm = rng.permutation(U)
        tied, strong, weak = perm[:300], perm[300:320], perm[320:2020]
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
        base[9, strong] *= 18.0 + np.arange(20)
        base[9, weak] *= 2.0
    elif case == "many_ties_at_cut":
        tied = rng.choice(U, 1500, replace=False)
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
    elif case == "huge_pool":
        U = 14000
        base = np.exp(rng.normal(scale=0.05, size=(T, U)))
        alpha = 0.4                                # every unit triggers: |C_t| = U > 12,288
    elif case == "pool_at_capacity":
        U = 13000
        base = np.exp(rng.normal(scale=0.01, size=(T, U)))   # no natural triggers
        base[9, :12288] *= 6.0                     # exactly 12,288 candidates at t = 10
    ora = Oracle(U, window=5, max_o=max_o, lock_len=2, eps=1e-12)
    dn = torch.empty(U, dtype=torch.float64, device="cuda")
    say("selection path:", case, "units", U)
    with Controller(U, 5, max_o, 2, 1e-12, np.zeros(U + 1), [], []) as ctl:
        for t in range(1, T + 1):
            dn.copy_(torch.from_numpy(base[t - 1]))
            ctl.step_from_norms(dn, alpha, 1.5)
            ref = ora.step(base[t - 1], alpha, 1.5)
            assert_step_matches(ctl.query(), ref, rtol=1e-14, what=f"{case} t={t}")
            if t == 10:
                want = {"pool_at_capacity": 12288, "pool_at_count_limit": 128,
                        "pool_over_count_limit": 129, "small_pool_ties_at_cut": 100,
                        "small_tie_in_radix": 400}
                if case in want:
                    assert ref.stats["n_cand"] == want[case]
                if case == "mid_pool_ties_at_cut":
                    assert 128 < ref.stats["n_cand"] <= 12288


@pytest.mark.parametrize("U", [1024, 1025])
@pytest.mark.parametrize("case", ["small_pool_ties_at_cut", "radix_ties_at_cut", "every_unit"])
def test_single_workgroup_selection_at_its_limit(U, case):
    """The selection inside the single-workgroup kernel (K2 and K3 in one
    launch, used up to 1,024 units) at its size limit, and one unit past it
    (K2, then K3): a pool of 100 with a 60-unit tie at the cut (direct
    counting), a pool of 700 with a 90-unit tie at the cut (radix select in
    LDS), and every unit a candidate (alpha = 0.4); the oracle's decisions
    bit for bit."""
    torch = require_gpu()
    from paper_2606_00539_amd import Controller

    rng = np.random.default_rng(U + len(case))
    T, max_o, alpha = 12, 64, 1.1
    base = np.exp(rng.normal(scale=0.01, size=(T, U)))       # no natural triggers
    perm = rng.permutation(U)
    if case == "small_pool_ties_at_cut":
        tied, strong, weak = perm[:60], perm[60:80], perm[80:100]
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
        base[9, strong] *= 18.0 + np.arange(20)
        base[9, weak] *= 2.0
    elif case == "radix_ties_at_cut":
        tied, strong, weak = perm[:90], perm[90:130], perm[130:700]
        base[:, tied] = base[:, tied[:1]]
        base[9, tied] *= 6.0
        base[9, strong] *= 18.0 + np.arange(40)
        base[9, weak] *= 2.0 + 0.01 * rng.random(570)
    else:
        alpha = 0.4                                          # |C_t| = U every step
    ora = Oracle(U, window=5, max_o=max_o, lock_len=2, eps=1e-12)
    dn = torch.empty(U, dtype=torch.float64, device="cuda")
    say("single-workgroup selection:", case, "units", U)
    with Controller(U, 5, max_o, 2, 1e-12, np.zeros(U + 1), [], []) as ctl:
        for t in range(1, T + 1):
            dn.copy_(torch.from_numpy(base[t - 1]))
            ctl.step_from_norms(dn, alpha, 1.5)
            ref = ora.step(base[t - 1], alpha, 1.5)
            assert_step_matches(ctl.query(), ref, rtol=1e-14, what=f"{case} U={U} t={t}")
            if t == 10 and case != "every_unit":
                assert ref.stats["n_cand"] == (100 if case == "small_pool_ties_at_cut" else 700)
            if case == "every_unit":
                assert ref.stats["n_cand"] == U


@pytest.mark.parametrize("name", ["tiny", "llama2-13b", "moe", "fine32"])
@pytest.mark.parametrize("policy", ["admitted", "warmup", "admitted_warmup", "admitted_alpha04"])
def test_policy_variants(name, policy):
    """The admitted-only budget (App. C budget-convention remark) and the
    high-fidelity warm-up (App. E.6) against the oracle, norm-level streams."""
    torch = require_gpu()
    from paper_2606_00539_amd import GNMR_BUDGET_ACTIVE, GNMR_BUDGET_ADMITTED, Controller

    w = R.get(name)
    norms = R.surrogate_norms(w, seed=3)
    mode = GNMR_BUDGET_ADMITTED if policy.startswith("admitted") else GNMR_BUDGET_ACTIVE
    warm = int(np.ceil(0.05 * w.steps)) if "warmup" in policy else 0
    alpha_of = (lambda t: 0.4) if policy.endswith("alpha04") else w.alpha
    say("policy:", name, policy, "warm-up", warm)
    ora = Oracle(w.num_units, window=w.window, max_o=w.max_o, lock_len=w.lock_len, eps=w.eps,
                 budget_mode=mode, warmup_steps=warm)
    dn = torch.empty(w.num_units, dtype=torch.float64, device="cuda")
    with Controller(w.num_units, w.window, w.max_o, w.lock_len, w.eps, np.zeros(w.num_units + 1),
                    [], [], budget_mode=mode, warmup_steps=warm) as ctl:
        for t in range(1, w.steps + 1):
            dn.copy_(torch.from_numpy(norms[t - 1]))
            ctl.step_from_norms(dn, alpha_of(t), w.beta(t))
            ref = ora.step(norms[t - 1], alpha_of(t), w.beta(t))
            assert_step_matches(ctl.query(), ref, rtol=1e-14, what=f"{name}/{policy} t={t}")


def test_state_roundtrip_admitted_keeps_previous_active_set():
    torch = require_gpu()
    from paper_2606_00539_amd import GNMR_BUDGET_ADMITTED, Controller

    w = R.get("fine128")
    norms = R.surrogate_norms(w)[:40]
    dn = torch.empty(w.num_units, dtype=torch.float64, device="cuda")
    mk = lambda: Controller(w.num_units, w.window, w.max_o, w.lock_len, w.eps,
                            np.zeros(w.num_units + 1), [], [], budget_mode=GNMR_BUDGET_ADMITTED)
    a, b = mk(), mk()
    for t in range(1, 21):
        dn.copy_(torch.from_numpy(norms[t - 1]))
        a.step_from_norms(dn, 0.9, 1.5)
    b.set_state(a.get_state())
    for t in range(21, 41):
        dn.copy_(torch.from_numpy(norms[t - 1]))
        a.step_from_norms(dn, 0.9, 1.5)
        b.step_from_norms(dn, 0.9, 1.5)
        qa, qb = a.query(), b.query()
        for f in ("mask", "lock", "norm", "gnmr", "dgnmr", "risk"):
            assert np.array_equal(qa[f], qb[f])
        assert qa["stats"] == qb["stats"]
    a.close()
    b.close()


@pytest.mark.parametrize("name", ["tiny", "llama2-13b", "moe", "fine32"])
def test_static_baseline(name):
    """ADAPT-style static baseline (App. E.4): profile W steps with every unit
    recovering, then fix the top-25% units by mean GNMR."""
    torch = require_gpu()
    from paper_2606_00539_amd import GNMR_BUDGET_STATIC, Controller

    w = R.get(name)
    norms = R.surrogate_norms(w, seed=5)
    W = max(1, int(np.ceil(0.05 * w.steps)))
    K = int(np.ceil(0.25 * w.num_units))
    say("static baseline:", name, "W", W, "K", K)
    ora = Oracle(w.num_units, window=w.window, max_o=K, lock_len=w.lock_len, eps=w.eps,
                 budget_mode=GNMR_BUDGET_STATIC, warmup_steps=W)
    dn = torch.empty(w.num_units, dtype=torch.float64, device="cuda")
    with Controller(w.num_units, w.window, K, w.lock_len, w.eps, np.zeros(w.num_units + 1),
                    [], [], budget_mode=GNMR_BUDGET_STATIC, warmup_steps=W) as ctl:
        for t in range(1, w.steps + 1):
            dn.copy_(torch.from_numpy(norms[t - 1]))
            ctl.step_from_norms(dn, w.alpha(t), w.beta(t))
            ref = ora.step(norms[t - 1], w.alpha(t), w.beta(t))
            assert_step_matches(ctl.query(), ref, rtol=1e-14, what=f"{name}/static t={t}")
            if t > W:
                assert ref.mask.sum() == K


def test_torch_units_on_a_model():
    """Gradients of a small LLaMA-style block stack registered by name; one
    unit per projection weight and one block-as-unit variant."""
    torch = require_gpu()
    from paper_2606_00539_amd.torch_units import TorchUnits, llama_linear_units

    torch.manual_seed(0)
    d, f = 96, 160

    def block():
        return torch.nn.ModuleDict({n: torch.nn.Linear(*s, bias=False) for n, s in (
            ("q_proj", (d, d)), ("k_proj", (d, d)), ("v_proj", (d, d)), ("o_proj", (d, d)),
            ("gate_proj", (d, f)), ("up_proj", (d, f)), ("down_proj", (f, d)))})

    model = torch.nn.ModuleDict({"layers": torch.nn.ModuleList([block(), block()])})
    model = model.to("cuda", torch.bfloat16)
    params = list(model.named_parameters())
    per_op = TorchUnits(params, max_o=2, lock_len=2, unit_of=llama_linear_units)
    per_block = TorchUnits(params, max_o=1, lock_len=2,
                           unit_of=lambda n: ".".join(n.split(".")[:2]))
    assert len(per_op.unit_names) == 14 and per_block.unit_names == ["layers.0", "layers.1"]
    ora_op = Oracle(14, window=5, max_o=2, lock_len=2, eps=1e-12)
    ora_blk = Oracle(2, window=5, max_o=1, lock_len=2, eps=1e-12)
    gen = torch.Generator(device="cuda").manual_seed(1)
    for t in range(1, 13):
        for i, (name, p) in enumerate(params):
            scale = 1e-3 * (20.0 if (t == 9 and i == 4) else 1.0)
            p.grad = (torch.randn(p.shape, device="cuda", generator=gen) * scale).to(p.dtype)
        per_op.step(1.1, 1.5)
        per_block.step(1.1, 1.5)
        host = {n: p.grad.view(torch.int16).cpu().numpy().view(np.uint16) for n, p in params}
        n_op = [oracle_norm([(host[n], 1)]) for n in per_op.param_names]
        n_blk = [oracle_norm([(host[n], 1) for n in per_block.param_names if n.startswith(u + ".")])
                 for u in per_block.unit_names]
        for ctl, ora, norms in ((per_op, ora_op, n_op), (per_block, ora_blk, n_blk)):
            ref = ora.step(norms, 1.1, 1.5)
            assert_step_matches(ctl.query(), ref, rtol=1e-5, what=f"torch units t={t}")
        if t == 9:   # the spiked projection and its block go to the recovery path
            assert "layers.0.gate_proj" in per_op.recovery_set()
            assert per_block.recovery_set() == ["layers.0"]
    per_op.close()
    per_block.close()


def test_graph_captured_step_replays_match_oracle(gen):
    """gnmr_step captured once in a HIP graph and replayed for the rest of
    the tiny stream; fresh gradients and synchronisations between replays;
    every replay checked against the oracle."""
    torch = require_gpu()
    w = R.get("tiny")
    nudge, _, ref, alphas, betas = S.guarded_stream(
        w, lambda t, s32, units: S.host_norms(w, t, s32, units))
    lay = L.for_workload(w)
    buf, base, ptrs = device_buffer(torch, lay)
    capture_at = 5
    assert len(set(alphas[capture_at - 1:])) == 1 and len(set(betas)) == 1
    with controller_for(lay, w, ptrs) as ctl:
        for t in range(1, capture_at):
            gen.fill(lay, base, w.seed, t, w.scale32(t, nudge[t - 1]))
            ctl.step(alphas[t - 1], betas[t - 1])
            assert_step_matches(ctl.query(), ref[t - 1], what=f"eager t={t}")
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        gen.fill(lay, base, w.seed, capture_at, w.scale32(capture_at, nudge[capture_at - 1]))
        torch.cuda.synchronize()
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                ctl.step(alphas[capture_at - 1], betas[capture_at - 1], stream=side)
        torch.cuda.synchronize()
        assert ctl.query()["stats"]["t"] == capture_at - 1   # capture ran nothing
        for t in range(capture_at, w.steps + 1):
            if t > capture_at:
                gen.fill(lay, base, w.seed, t, w.scale32(t, nudge[t - 1]))
            graph.replay()
            torch.cuda.synchronize()
            assert_step_matches(ctl.query(), ref[t - 1], what=f"replay t={t}")
