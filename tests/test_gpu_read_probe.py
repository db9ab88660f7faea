"""The benchmark's read-ceiling probes (synth library) read every 16-byte
word of the buffer exactly once: on words of 1.0f the partials sum to
4 x the number of words, for sizes that end inside a block, a grid stride
and an unrolled round."""
import numpy as np
import pytest

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nvec", [1, 4095, 4096, 4097, 2048 * 256 * 8 + 3, 3_000_017])
def test_read_probe_reads_every_word_once(nvec):
    torch = require_gpu()
    from synth.gpu import ReadProbe

    rp = ReadProbe()
    buf = torch.ones(nvec * 4 + 64, dtype=torch.float32, device="cuda")
    buf[nvec * 4:] = 1e6          # past the end: must not be read
    for v in rp.VARIANTS:
        parts = torch.full((rp.num_partials(nvec * 16, v),), float("nan"), device="cuda")
        rp.run(buf.data_ptr(), nvec * 16, parts.data_ptr(), v)
        torch.cuda.synchronize()
        got = parts.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(got)), f"variant {v}: partial not written"
        assert got.sum() == 4.0 * nvec, f"variant {v}: {got.sum()} != {4 * nvec}"


def test_read_probe_rejects_bad_arguments():
    torch = require_gpu()
    from synth.gpu import ReadProbe

    rp = ReadProbe()
    buf = torch.ones(64, dtype=torch.float32, device="cuda")
    parts = torch.zeros(4096, dtype=torch.float32, device="cuda")
    for ptr, n, v in [(buf.data_ptr() + 4, 64, 1), (buf.data_ptr(), 60, 0),
                      (buf.data_ptr(), 64, 2), (0, 64, 0)]:
        with pytest.raises(RuntimeError):
            rp.run(ptr, n, parts.data_ptr(), v)


@pytest.mark.parametrize("nvec", [1, 1023, 1024, 1025, 3_000_017])
def test_copy_probe_copies_exactly(nvec):
    torch = require_gpu()
    from synth.gpu import ReadProbe

    rp = ReadProbe()
    src = torch.arange(nvec * 4, dtype=torch.int32, device="cuda")
    dst = torch.full((nvec * 4 + 64,), -1, dtype=torch.int32, device="cuda")
    rp.copy(src.data_ptr(), dst.data_ptr(), nvec * 16)
    torch.cuda.synchronize()
    assert torch.equal(dst[:nvec * 4], src)
    assert bool((dst[nvec * 4:] == -1).all()), "copied past the end"
