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


def test_golden_net_weights_match_the_library_draw():
    """The full-batch network digests were written from weights drawn by the
    digest script itself (oracle layouts); the GPU test rebuilds them with
    the library's synthetic_weights (its layouts).  Both must be the same
    tensors, zeroed filters and exponents included."""
    import importlib.util
    import os
    from paper_2009_13108_amd import model as M
    path = os.path.join(os.path.dirname(__file__), "golden", "make_fullsize.py")
    spec = importlib.util.spec_from_file_location("make_fullsize", path)
    mk = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mk)
    cases = [(M.LENET5, 1, M.LENET5_REAL["zero_filters"], 40)]
    cases += [(M.vgg_small(d), 3, {}, 34 + d) for d in (7, 8, 9)]
    for specs, img_c, zf, cfg in cases:
        wo, eo = mk.net_weights(specs, cfg, img_c, zf)
        wl, el = M.synthetic_weights(specs, 4, cfg, image_channels=img_c, zero_filters=zf)
        assert eo == el
        for a, b in zip(wo, wl):
            assert (mk.nhwc(a) == b).all() if a.ndim == 4 else (a == b).all()
