"""The allocation-free gradient pass (gnmr_sumsq_noalloc, through the C ABI)
against the context-based one (gnmr_sumsq) and the oracle: two calls in a
row on one device, the second over a smaller layout, each bit-identical to
gnmr_sumsq over the same layout and within the fp32-accumulation bar of the
oracle's float64 sum of squares."""
import sys

import numpy as np
import pytest

from gpu_util import controller_for, device_buffer, require_gpu
from oracle import sumsq as oracle_sumsq
from synth import layout as L
from synth import values as V

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def layout(sizes, dtypes, rng):
    pieces, shift = [], []
    for b, n in enumerate(sizes):
        if n > 20 and b % 3 == 0:
            cut = int(rng.integers(1, n))
            p = [cut, 0, n - cut]                      # with an empty segment
        else:
            p = [n] if n > 0 else []
        pieces.append(p)
        esz = V.DTYPE_SIZE[dtypes[b]]
        shift += [int(rng.integers(0, 16 // esz)) * esz for _ in p]
    return L.build(sizes, dtypes, pieces=pieces, shift=shift), pieces


def oracle_unit(seed, t, b, scale, dtype, pieces):
    segs, start = [], 0
    for m in pieces:
        segs.append((V.unit_values(seed, t, b, scale, dtype, start, m), dtype))
        start += m
    return oracle_sumsq(segs)


def run_case(torch, gen, sizes, dtypes, seed, t):
    from paper_2606_00539_amd import gnmr_sumsq_noalloc

    rng = np.random.default_rng(seed)
    lay, pieces = layout(sizes, dtypes, rng)
    U = lay.num_units
    say(f"no-alloc sumsq: {U} units, {lay.num_segments} segments, {lay.total_bytes} bytes")
    buf, base, ptrs = device_buffer(torch, lay)
    scale = (10.0 ** rng.uniform(-4, -2, size=U)).astype(np.float32)
    gen.fill(lay, base, seed, t, scale)
    got = torch.full((U,), -1.0, dtype=torch.float64, device="cuda")
    gnmr_sumsq_noalloc(U, lay.unit_seg_off, lay.seg_numel, lay.seg_dtype, ptrs, got)
    want = torch.zeros(U, dtype=torch.float64, device="cuda")
    with controller_for(lay, ptrs=ptrs, window=5, max_o=2, lock_len=1, eps=0.0) as ctl:
        ctl.sumsq(want)
    torch.cuda.synchronize()
    g, w = got.cpu().numpy(), want.cpu().numpy()
    assert np.array_equal(g.view(np.uint64), w.view(np.uint64)), np.flatnonzero(g != w)[:10]
    for b in range(U):
        ref = oracle_unit(seed, t, b, float(scale[b]), dtypes[b], pieces[b])
        if sizes[b] == 0:
            assert g[b] == 0.0
        else:
            assert abs(g[b] - ref) <= 5e-6 * ref, (b, sizes[b], g[b], ref)
    del buf


def test_noalloc_sumsq_matches_context_pass_twice_then_smaller():
    torch = require_gpu()
    from synth.gpu import Generator

    gen = Generator()
    big = [0, 1, 7, 9, 4095, 32767, 32769, 65536 * 3 + 5, 1_000_003, 123_457, 2, 4_000_001,
           700_001, 16_384, 16_385]
    dt_big = [i % 2 for i in range(len(big))]
    run_case(torch, gen, big, dt_big, seed=31, t=1)
    small = [5, 33_333, 0, 100_000]
    run_case(torch, gen, small, [1, 0, 1, 0], seed=32, t=2)


def test_noalloc_sumsq_refuses_a_layout_beyond_its_scratch():
    torch = require_gpu()
    from paper_2606_00539_amd import GnmrError, gnmr_sumsq_noalloc
    from paper_2606_00539_amd import binding as B

    # 2^21 bf16 items of 64 KiB: 40 MiB of work list and partials.  The
    # call is refused before any device work, so the segment pointer is
    # never dereferenced.
    n = (1 << 21) * 32768
    out = torch.zeros(1, dtype=torch.float64, device="cuda")
    with pytest.raises(GnmrError) as e:
        gnmr_sumsq_noalloc(1, [0, 1], [n], [B.GNMR_BF16], [1 << 20], out)
    assert e.value.status == B.GNMR_E_INVALID and "scratch" in str(e.value)
