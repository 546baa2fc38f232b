"""The seeded input generator gives identical bytes on the host (numpy) and
through torch (CPU here; the GPU case is in test_gpu_fullsize)."""
import numpy as np
import pytest

from paper_2009_13108_amd import inputs as I


@pytest.mark.parametrize("lo,hi,dt", [(-127, 127, np.int8), (0, 127, np.int8), (-15, 15, np.int8),
                                      (0, 255, np.uint8), (0, 999, np.int32),
                                      (-(1 << 29), 1 << 29, np.int32)])
def test_torch_stream_matches_numpy(lo, hi, dt):
    a = I.uniform_int(12345, (1000, 37), lo, hi, dtype=dt)
    b = I.uniform_int(12345, (1000, 37), lo, hi, dtype=dt, device="cpu").numpy()
    assert a.dtype == b.dtype and (a == b).all()
    assert a.min() >= lo and a.max() <= hi


def test_distribution_is_flat():
    a = I.weights(7, (1 << 20,)).astype(np.int64)
    h = np.bincount(a + 127, minlength=255)
    assert h.min() > 0.9 * h.mean() and h.max() < 1.1 * h.mean()
