"""The C-ABI library loads on a host without a GPU, exports every entry point
that include/gnmr.h declares, and rejects bad configurations before touching
the device.  CPU only."""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_entry_points():
    text = open(os.path.join(ROOT, "include", "gnmr.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gnmr_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_entry_points()
    for n in ("gnmr_init", "gnmr_step", "gnmr_query", "gnmr_destroy", "gnmr_step_from_norms",
              "gnmr_get_state", "gnmr_set_state", "gnmr_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2606_00539_amd import binding as B

    lib = B.load_library()
    missing = [n for n in declared_entry_points() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(B.EXPORTED) == set(declared_entry_points())


def test_struct_layouts_match_header():
    import ctypes

    from paper_2606_00539_amd import binding as B

    assert ctypes.sizeof(B.gnmr_config) == 40
    assert ctypes.sizeof(B.gnmr_segments) == 40
    assert ctypes.sizeof(B.gnmr_stats) == 40
    assert ctypes.sizeof(B.gnmr_wgrad_problem) == 48


@pytest.mark.parametrize("bad", [
    dict(num_units=0), dict(window=0), dict(max_o=-1), dict(lock_len=-2), dict(eps=-1.0),
    dict(eps=float("nan")), dict(unit_seg_off=[0, 2, 1]), dict(unit_seg_off=[1, 1, 1]),
    dict(seg_numel=[-1]), dict(seg_dtype=[7]), dict(budget_mode=3), dict(warmup_steps=-1),
    dict(budget_mode=2, warmup_steps=0),
    dict(seg_numel=[(1 << 50) + 1]),                     # above 2^50 elements
    dict(seg_numel=[16777215 * 32768 + 1]),              # one bf16 item too many
])
def test_init_rejects_bad_configuration(bad):
    from paper_2606_00539_amd import GnmrError, gnmr_init
    from paper_2606_00539_amd import binding as B

    args = dict(num_units=2, window=5, max_o=1, lock_len=1, eps=0.0,
                unit_seg_off=[0, 1, 1], seg_numel=[10], seg_dtype=[B.GNMR_BF16])
    args.update(bad)
    if "unit_seg_off" in bad and bad["unit_seg_off"][-1] != 1:
        args["num_units"] = len(bad["unit_seg_off"]) - 1
    with pytest.raises(GnmrError) as e:
        gnmr_init(**args)
    assert e.value.status == B.GNMR_E_INVALID
    assert B.gnmr_last_error() != ""


@pytest.mark.parametrize("bad", [
    dict(cols=12), dict(cols=0), dict(cols=16392), dict(unit=5), dict(unit=-1), dict(rows=-1),
    dict(in_=8), dict(out=0),
])
def test_actuator_rejects_bad_segments(bad):
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    seg = dict(in_=4096, out=8192, rows=4, cols=64, unit=1)
    seg.update(bad)
    with pytest.raises(GnmrError) as e:
        B.gnmr_actuator_create([(seg["in_"], seg["out"], seg["rows"], seg["cols"], seg["unit"])],
                               num_units=5)
    assert e.value.status == B.GNMR_E_INVALID


# in [4096, 4608) out [8192, 8704) for 4 rows of 64 features; each case's
# segments are rejected in the argument checks, before any device call
_A = (4096, 8192, 4, 64, 0)


@pytest.mark.parametrize("segs", [
    [(4096, 4096 + 256, 4, 64, 0)],                      # out partly overlaps its own in
    [_A, (8192, 12288, 4, 64, 1)],                       # reads another segment's output
    [_A, (12288, 8192 + 256, 4, 64, 1)],                 # outputs overlap
    [(4096, 4096, 4, 64, 0), (4096, 12288, 4, 64, 1)],   # in place over another's input
    [(8192, 8192, 4, 64, 0), (8128, 32768, 1, 40, 1)],   # in place over the tail of an input
    [(20480, 20480, 4, 64, 0), (12288, 16384, 4, 64, 1), (16384 + 496, 24576, 1, 8, 2)],
])
def test_actuator_rejects_racing_segments(segs):
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    with pytest.raises(GnmrError) as e:
        B.gnmr_actuator_create(segs, num_units=3)
    assert e.value.status == B.GNMR_E_INVALID
    assert "overlap" in B.gnmr_last_error()


def _races(segs):
    """Brute force over every pair: a write that meets another write, another
    segment's input, or its own input other than exactly (in place)."""
    span = [(i, i + r * c * 2, o, o + r * c * 2) for i, o, r, c, _ in segs if r > 0]
    meet = lambda a0, a1, b0, b1: a0 < b1 and b0 < a1  # noqa: E731
    for k, (i0, i1, o0, o1) in enumerate(span):
        if o0 != i0 and meet(o0, o1, i0, i1):
            return True
        for j, (j0, j1, p0, p1) in enumerate(span):
            if j != k and (meet(o0, o1, j0, j1) or meet(o0, o1, p0, p1)):
                return True
    return False


@pytest.mark.parametrize("segs", [
    [(1 << 40, 2 << 40, 4 * 16777215 + 1, 8, 0)],
    [(1 << 40, 2 << 40, 3 * 16777215, 8, 0), (3 << 40, 4 << 40, 16777216, 8, 1)],
    [(1 << 40, 2 << 40, 16777216, 4104, 0)],
])
def test_actuator_rejects_more_rows_than_one_launch_holds(segs):
    # the limit is checked before any allocation or device call
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    with pytest.raises(GnmrError) as e:
        B.gnmr_actuator_create(segs, num_units=2)
    assert e.value.status == B.GNMR_E_INVALID and "one launch" in B.gnmr_last_error()


def test_actuator_overlap_check_equals_brute_force():
    # random layouts of fake addresses; a layout without a race passes the
    # checks and fails only later, at the table allocation (no device here),
    # or succeeds where there is one (the tables hold only the addresses)
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    rng = np.random.default_rng(77)
    seen = {True: 0, False: 0}
    for _ in range(400):
        n = int(rng.integers(1, 7))
        segs = []
        for _ in range(n):
            i = 4096 + 16 * int(rng.integers(0, 400))
            o = i if rng.random() < 0.3 else 4096 + 16 * int(rng.integers(0, 400))
            segs.append((i, o, int(rng.integers(0, 3)), 8 * int(rng.integers(1, 9)),
                         int(rng.integers(0, 3))))
        want = _races(segs)
        seen[want] += 1
        try:
            act = B.gnmr_actuator_create(segs, num_units=3)
        except GnmrError as e:
            assert (e.status == B.GNMR_E_INVALID) == want, (segs, B.gnmr_last_error())
        else:
            assert not want, segs
            B.gnmr_actuator_destroy(act)
    assert seen[True] > 50 and seen[False] > 50


@pytest.mark.parametrize("bad", [
    dict(cols=12), dict(cols=0), dict(cols=16392), dict(rows=-1), dict(rows=1 << 31),
    dict(unit=-1), dict(fmt_low=6), dict(fmt_rec=-1), dict(x=4096 + 8), dict(out=8192 + 2),
    dict(rows=4 * 16777215 + 1, cols=8), dict(rows=16777216, cols=4104),
    dict(x=0), dict(mask=0), dict(out=4096 + 16), dict(x=8192 - 16),
])
def test_actuate_matrix_rejects_bad_arguments(bad):
    # in [4096, 4608), out [8192, 8704): every case fails in the argument
    # checks, before any device call
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    a = dict(x=4096, out=8192, rows=4, cols=64, mask=65536, unit=3, fmt_low=1, fmt_rec=0)
    a.update(bad)
    with pytest.raises(GnmrError) as e:
        B.gnmr_actuate_matrix(a["x"], a["out"], a["rows"], a["cols"], a["mask"], a["unit"],
                              a["fmt_low"], a["fmt_rec"])
    assert e.value.status == B.GNMR_E_INVALID


def test_actuate_matrix_with_no_rows_launches_nothing():
    # rows = 0 returns before any device call, whatever the pointers
    from paper_2606_00539_amd import binding as B

    B.gnmr_actuate_matrix(0, 0, 0, 64, 0, 0, 1, 0)


def test_missing_library_fails_loudly(tmp_path):
    from paper_2606_00539_amd import binding as B

    with pytest.raises(RuntimeError, match="not built"):
        B.load_library(str(tmp_path / "libgnmr.so"))


def test_bench_refuses_more_than_one_gpu():
    import subprocess
    import sys

    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "8"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


@pytest.mark.parametrize("bad", [
    dict(out_f=12), dict(in_f=4), dict(out_f=0), dict(in_f=-8), dict(tokens=-1),
    dict(dy=0), dict(x=0), dict(dw=0), dict(ss=0), dict(dy=4096 + 8), dict(dw=8192 + 2),
    dict(in_f=1 << 24), dict(out_f=1 << 24), dict(out_f=1 << 20, in_f=1 << 20),
])
def test_wgrad_rejects_bad_arguments(bad):
    # every case fails in the argument checks, before any device call
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    a = dict(dy=4096, x=8192, dw=16384, tokens=16, out_f=64, in_f=128, ss=32768)
    a.update(bad)
    with pytest.raises(GnmrError) as e:
        B.gnmr_wgrad_sumsq(a["dy"], a["x"], a["dw"], a["tokens"], a["out_f"], a["in_f"], a["ss"])
    assert e.value.status == B.GNMR_E_INVALID


def test_wgrad_tile_count():
    from paper_2606_00539_amd import gnmr_wgrad_num_tiles

    assert gnmr_wgrad_num_tiles(5120, 5120) == 400
    assert gnmr_wgrad_num_tiles(13824, 5120) == 54 * 20
    assert gnmr_wgrad_num_tiles(264, 520) == 2 * 3
    assert gnmr_wgrad_num_tiles(0, 8) == 0


def test_wgrad_batched_rejects_a_bad_problem_before_launching():
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    good = (4096, 8192, 16384, 16, 64, 128)
    bad = (4096, 8192, 16384, 16, 60, 128)
    with pytest.raises(GnmrError) as e:
        B.gnmr_wgrad_sumsq_batched([good, bad], 32768)
    assert e.value.status == B.GNMR_E_INVALID
    with pytest.raises(GnmrError):
        B.gnmr_wgrad_sumsq_batched([good], 0)


@pytest.mark.parametrize("probs,ss", [
    ([(4096, 8192, 4096, 16, 64, 128)], 65536),                  # dw over its own dy
    ([(4096, 8192, 16384, 16, 64, 128)], 16384 + 4096),          # tile sums inside dw
    ([(4096, 8192, 16384, 16, 64, 128), (40960, 45056, 16384 + 8192, 16, 64, 128)], 65536),
    ([(4096, 8192, 16384, 16, 64, 128), (40960, 16384 + 512, 49152, 16, 64, 128)], 65536),
    ([(4096, 8192, 16384, 16, 64, 128), (32768, 49152, 12288 - 16, 16, 16, 128)], 65536),
])
def test_wgrad_batched_rejects_racing_outputs(probs, ss):
    # outputs that overlap another buffer of the batch; checked before launching
    from paper_2606_00539_amd import GnmrError
    from paper_2606_00539_amd import binding as B

    with pytest.raises(GnmrError) as e:
        B.gnmr_wgrad_sumsq_batched(probs, ss)
    assert e.value.status == B.GNMR_E_INVALID
    assert "overlap" in B.gnmr_last_error()


def test_wgrad_batched_rejects_nonzero_reserved():
    import ctypes

    from paper_2606_00539_amd import binding as B

    p = B.gnmr_wgrad_problem(4096, 8192, 16384, 16, 64, 128, 0, 7)
    st = B.load_library().gnmr_wgrad_sumsq_batched(ctypes.byref(p), 1, 32768, None)
    assert st == B.GNMR_E_INVALID and "reserved" in B.gnmr_last_error()


def test_fused_wgrad_units_rejects_unsupported_layers():
    # argument checks before any device work: fp32 or host weights, odd shapes
    import torch

    from paper_2606_00539_amd.torch_units import FusedWgradUnits

    with pytest.raises(TypeError):
        FusedWgradUnits([("a", torch.nn.Linear(16, 16, bias=False))])
    with pytest.raises(ValueError):
        FusedWgradUnits([])


def test_per_token_quantisation_refuses_other_element_types():
    # the kernel reads bf16 rows: an fp32 or host tensor is refused before any
    # library call (an fp32 buffer would otherwise be misread as bf16)
    import torch

    from paper_2606_00539_amd.torch_units import _quantize_rows

    spec = (1 << 20, 0, 1, 3)               # never dereferenced
    with pytest.raises(TypeError, match="bf16"):
        _quantize_rows(torch.zeros(4, 16, dtype=torch.float32), spec)
    with pytest.raises(TypeError, match="HIP device"):
        _quantize_rows(torch.zeros(4, 16, dtype=torch.bfloat16), spec)


def test_noalloc_sumsq_rejects_bad_arguments_before_the_device():
    """gnmr_sumsq_noalloc checks the layout, the pointers and the scratch size
    on the host; none of these calls reaches the device (the pointers are
    never dereferenced)."""
    from paper_2606_00539_amd import GnmrError, gnmr_sumsq_noalloc
    from paper_2606_00539_amd import binding as B

    out = 1 << 24
    cases = [
        (0, [0], [], [], [], out),                                  # no unit
        (2, [0, 1, 1], [10], [B.GNMR_BF16], None, out),             # pointers required
        (1, [0, 1], [10], [B.GNMR_BF16], [0], out),                 # NULL segment pointer
        (1, [0, 1], [10], [B.GNMR_F32], [(1 << 20) + 2], out),      # misaligned fp32
        (1, [0, 1], [10], [7], [1 << 20], out),                     # unknown dtype
        (1, [0, 1], [10], [B.GNMR_BF16], [1 << 20], 0),             # no output
        # 2^21 bf16 items: work list and partials beyond the 32 MiB scratch
        (1, [0, 1], [(1 << 21) * 32768], [B.GNMR_BF16], [1 << 20], out),
    ]
    for U, off, numel, dt, ptrs, d_out in cases:
        with pytest.raises(GnmrError) as e:
            gnmr_sumsq_noalloc(U, off, numel, dt, ptrs, d_out)
        assert e.value.status == B.GNMR_E_INVALID, (U, off, numel, dt, ptrs)
    assert B.GNMR_NOALLOC_SCRATCH_BYTES == 32 << 20
