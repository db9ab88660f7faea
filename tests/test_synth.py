"""The seeded input generator (host twin): determinism, rounding, moments,
workload shapes."""
import numpy as np
import pytest
import torch

from synth import recipe as R
from synth import values as V


def test_mix64_matches_python_ints():
    xs = np.array([0, 1, 2, 0xDEADBEEF, (1 << 64) - 1, V.GAMMA], dtype=np.uint64)
    got = V.mix64_np(xs.copy())
    for x, g in zip(xs.tolist(), got.tolist()):
        assert V.mix64_int(int(x)) == g


def test_splitmix64_reference_sequence():
    # SplitMix64 seeded with 1234567: published first outputs of the generator
    # (state += GAMMA; output = mix64(state)).
    state = 1234567
    outs = []
    for _ in range(3):
        state = (state + V.GAMMA) & V.MASK64
        outs.append(V.mix64_int(state))
    assert outs == [6457827717110365317, 3203168211198807973, 9817491932198370423]


def test_bf16_rounding_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = (rng.normal(size=100000) * 10.0 ** rng.uniform(-8, 3, size=100000)).astype(np.float32)
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0]   # exact ties
    ours = V.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_values_are_counter_based():
    a = V.unit_values(0, 3, 5, 1e-3, V.DTYPE_BF16, 0, 1000)
    b = V.unit_values(0, 3, 5, 1e-3, V.DTYPE_BF16, 400, 600)
    assert np.array_equal(a[400:], b)
    c = V.unit_values(0, 4, 5, 1e-3, V.DTYPE_BF16, 0, 1000)
    assert not np.array_equal(a, c)


def test_table_and_moments():
    z = V.normal_table()
    assert z.shape == (65536,) and z.dtype == np.float32
    assert np.array_equal(z, -z[::-1])                      # symmetric quantiles
    x = V.unit_values(0, 1, 0, 1.0, V.DTYPE_F32, 0, 1 << 20)
    assert abs(x.mean()) < 5e-3 and abs(x.var() - 1.0) < 5e-3


@pytest.mark.parametrize("name,units,numel,nbytes", [
    ("tiny", 28, 3_162_112, 12_648_448),
    ("llama2-7b", 224, 6_476_005_376, 12_952_010_752),
    ("llama2-13b", 280, 12_687_769_600, 25_375_539_200),
    ("llama2-13b-layers", 40, 12_687_769_600, 25_375_539_200),
    ("moe", 5454, 15_868_624_896, 63_474_499_584),
    ("fine128", 10624, 6_476_005_376, 12_952_010_752),
    ("fine32", 42496, 6_476_005_376, 12_952_010_752),
])
def test_workload_shapes(name, units, numel, nbytes):
    w = R.get(name)
    assert w.num_units == units
    assert int(w.numel.sum()) == numel
    assert w.bytes_per_step == nbytes
    assert w.scale64.shape == (w.steps, units)
    assert np.all(np.isfinite(w.scale64)) and np.all(w.scale64 >= 0)


def test_two_stage_alpha():
    assert [R.two_stage_alpha(t, 16) for t in (1, 2)] == [1.5, 1.1]
    assert [R.two_stage_alpha(t, 256) for t in (7, 8)] == [1.5, 1.1]


@pytest.mark.parametrize("start,count", [(0, 1), (1, 7), (3, 4), (5, 1000), (1 << 20, 33)])
def test_table_indices_match_definition(start, count):
    # j(i) = (mix64(key + (i // 4 + 1) * GAMMA) >> (16 * (i % 4))) & 0xFFFF
    key = V.unit_key(7, 9, 11)
    want = [(V.mix64_int(key + (i // 4 + 1) * V.GAMMA) >> (16 * (i % 4))) & 0xFFFF
            for i in range(start, start + count)]
    assert V.table_indices(7, 9, 11, start, count).tolist() == want


def test_unit_values_chunking_is_seamless():
    a = V.unit_values(1, 2, 3, 5e-3, V.DTYPE_BF16, 5, 10_001, chunk=1 << 22)
    b = V.unit_values(1, 2, 3, 5e-3, V.DTYPE_BF16, 5, 10_001, chunk=999)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("dtype", [V.DTYPE_F32, V.DTYPE_BF16])
@pytest.mark.parametrize("start,count", [(0, 1), (2, 9), (7, 100_003), (1 << 24, 4)])
def test_c_twin_is_bit_identical(dtype, start, count):
    from synth import host

    a = V.unit_values(3, 17, 123, 7.7e-4, dtype, start, count)
    b = host.unit_values(3, 17, 123, 7.7e-4, dtype, start, count)
    assert a.dtype == b.dtype and np.array_equal(a, b)
