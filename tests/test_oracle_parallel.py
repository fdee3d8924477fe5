"""The oracle's process-parallel drivers against the oracle itself: the
band-parallel inference equals ``oracle.infer`` (up to the rounding order of
float64 matrix products; in practice bit for bit), and the parallel
light-cone windows equal ``oracle.infer_window`` per box."""
import os
import tempfile

import numpy as np
import pytest

import oracle
import oracle.parallel as par
from synthetic import Workload, make_image, make_weights, storage_dtype


def kw(wl):
    return dict(ndim=wl.ndim, n_in=wl.n_in, channels=wl.channels, factors=wl.factors,
                steps=wl.steps, fire_rate=wl.fire_rate, seed=wl.seed, dtype=storage_dtype(wl))


CASES = [
    Workload(name="banded_2d", ndim=2, extent=(1, 40, 56), n_in=3, factors=((1, 2, 2),),
             steps=(4, 3), image_kind="uniform"),
    Workload(name="banded_3d_f16", ndim=3, extent=(6, 20, 24), n_in=3,
             factors=((1, 2, 2),), steps=(3, 2), dtype="f16", image_kind="uniform"),
    Workload(name="banded_3d_nin1", ndim=3, extent=(5, 18, 16), n_in=1,
             factors=((1, 2, 2),), steps=(2, 2), image_kind="uniform"),
]


@pytest.mark.parametrize("wl", CASES, ids=lambda w: w.name)
def test_infer_banded_equals_infer(wl, monkeypatch):
    monkeypatch.setattr(par, "_MIN_PARALLEL_CELLS", 0)   # every level in bands
    image, weights = make_image(wl), make_weights(wl)
    want, want_seg = oracle.infer(image, weights, **kw(wl))
    got, got_seg = par.infer_banded(image, weights, workers=3, **kw(wl))
    assert got.dtype == want.dtype
    scale = float(np.max(np.abs(want.astype(np.float64))))
    assert float(np.max(np.abs(got.astype(np.float64) - want))) <= 1e-6 * scale
    assert np.mean(got_seg == want_seg) >= 0.999


def test_infer_banded_batch_index_reaches_the_mask(monkeypatch):
    monkeypatch.setattr(par, "_MIN_PARALLEL_CELLS", 0)
    wl = CASES[0]
    image, weights = make_image(wl), make_weights(wl)
    want, _ = oracle.infer(image, weights, batch=2, **kw(wl))
    got, _ = par.infer_banded(image, weights, workers=2, batch=2, **kw(wl))
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-6 * float(np.max(np.abs(want))))


def test_infer_windows_equal_infer_window():
    wl = CASES[1]
    image, weights = make_image(wl), make_weights(wl)
    boxes = [((0, 2), (0, 4), (0, 5)), ((4, 6), (16, 20), (19, 24)), ((2, 3), (7, 12), (9, 14))]
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "image.npy")
        np.save(path, image)
        got = par.infer_windows(path, weights, boxes, workers=2, **kw(wl))
    for box, g in zip(boxes, got):
        want = oracle.infer_window(image, weights, box, **kw(wl))
        np.testing.assert_array_equal(g, want)
