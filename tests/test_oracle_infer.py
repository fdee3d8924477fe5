"""Pins for the oracle's whole inference, its readout and its light-cone windows.

* the learnable parameters the oracle actually uses reproduce the parameter
  counts printed in the paper (tests/golden/paper_param_counts.json): per
  level, conv weights and bias, first linear with bias, and a second linear
  without bias producing only the hidden channels;
* whole inference equals a brute-force cell-by-cell pipeline on tiny grids
  (2D, 3D, anisotropic pooling, fp16 storage);
* the light-cone window evaluation equals the full-grid result cropped;
* readout is the two-class argmax with ties to the lower channel; the K-class
  readout is numpy's argmax over the last K channels (and the two-class
  readout for K = 2);
* the first-level step rule alpha0 * max(H, W, D) gives, on the paper's level
  table, the max(H, W) / 2^L steps named in Sec. 3.2.
"""
import json
import os

import numpy as np
import pytest

from oracle import (infer, infer_window, readout, readout_classes, first_level_steps,
                    InferLog)
from synthetic import (make_image, make_weights, scaled, TINY_2D, VOLUME_3D, VIDEO_2DT,
                       PATHOLOGY_184MP, Workload)

from brute import brute_infer

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run(wl, image=None, weights=None):
    image = make_image(wl) if image is None else image
    weights = make_weights(wl) if weights is None else weights
    dt = np.float16 if wl.dtype == "f16" else np.float32
    return infer(image, weights, ndim=wl.ndim, n_in=wl.n_in, channels=wl.channels,
                 factors=wl.factors, steps=wl.steps, fire_rate=wl.fire_rate, seed=wl.seed, dtype=dt)


def used_parameters(w, n_in):
    return w.conv_w.size + w.conv_b.size + w.w1.size + w.b1.size + w.w2[n_in:].size


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLDEN, "paper_param_counts.json")))["cases"])
def test_parameter_counts_match_paper(case):
    extent = (8, 8, 8) if case["ndim"] == 3 else (1, 8, 8)
    wl = Workload(name="count", ndim=case["ndim"], extent=extent, n_in=case["n_in"],
                  factors=((1, 1, 1),) * (case["levels"] - 1), steps=(1,) * case["levels"])
    ws = make_weights(wl)
    assert sum(used_parameters(w, wl.n_in) for w in ws) == case["params"]
    assert wl.params_per_level() * wl.levels == case["params"]


def test_oracle_uses_exactly_the_counted_parameters():
    """Changing an unused second-layer row (input channel) changes nothing;
    changing any counted parameter changes the output."""
    wl = scaled(TINY_2D, (1, 16, 16), steps=(2, 2, 2))
    img = make_image(wl)
    base, _ = run(wl, img)
    ws = make_weights(wl)
    ws[0].w2[: wl.n_in] += 1.0
    same, _ = run(wl, img, ws)
    np.testing.assert_array_equal(same, base)
    for name, sl in (("conv_w", (5, 4)), ("conv_b", (7,)), ("w1", (3, 20)), ("b1", (9,)),
                     ("w2", (wl.n_in + 1, 11))):
        ws = make_weights(wl)
        getattr(ws[0], name)[sl] += 0.5
        other, _ = run(wl, img, ws)
        assert np.abs(other - base).max() > 0, name


CASES = [
    scaled(TINY_2D, (1, 8, 12), steps=(2, 2, 3)),
    scaled(VOLUME_3D, (2, 8, 8), steps=(2, 1, 2)),
    Workload(name="aniso", ndim=3, extent=(4, 4, 8), n_in=3, factors=((2, 1, 2), (1, 2, 2)),
             steps=(1, 2, 2), image_kind="uniform"),
    scaled(VIDEO_2DT, (4, 8, 8), steps=(1, 1, 1, 1, 2), factors=((1, 2, 2), (1, 2, 2), (2, 1, 1), (2, 1, 1)),
           image_kind="uniform"),
]


@pytest.mark.parametrize("wl", CASES, ids=lambda w: w.name)
def test_infer_matches_brute_force(wl):
    img = make_image(wl)
    ws = make_weights(wl)
    dt = np.float16 if wl.dtype == "f16" else np.float32
    got_s, got_seg = run(wl, img, ws)
    want_s, want_seg = brute_infer(img, ws, wl.ndim, wl.n_in, wl.factors, wl.steps,
                                   wl.fire_rate, wl.seed, dt)
    assert got_s.dtype == dt
    if dt == np.float32:
        np.testing.assert_allclose(got_s, want_s, rtol=1e-6, atol=1e-6)
    else:
        np.testing.assert_allclose(got_s.astype(np.float32), want_s.astype(np.float32),
                                   rtol=2e-3, atol=2e-3)
    np.testing.assert_array_equal(got_s[..., :wl.n_in], img)


WINDOW_CASES = [
    (scaled(TINY_2D, (1, 64, 48), steps=(3, 4, 5)), [((0, 1), (0, 5), (0, 7)), ((0, 1), (20, 29), (13, 19)),
                                                      ((0, 1), (60, 64), (40, 48))]),
    (scaled(VOLUME_3D, (6, 16, 16), steps=(2, 3, 2)), [((0, 2), (0, 3), (5, 9)), ((2, 5), (7, 12), (7, 10))]),
    (scaled(VIDEO_2DT, (8, 16, 16), steps=(2, 1, 2, 1, 3)), [((3, 5), (4, 9), (10, 16))]),
    (scaled(PATHOLOGY_184MP, (1, 64, 96), steps=(2,) * 6, image_kind="blobs"),
     [((0, 1), (0, 4), (90, 96)), ((0, 1), (30, 35), (40, 43))]),
]


@pytest.mark.parametrize("wl,boxes", WINDOW_CASES, ids=lambda x: getattr(x, "name", "boxes"))
def test_window_equals_full_grid(wl, boxes):
    img = make_image(wl)
    ws = make_weights(wl)
    dt = np.float16 if wl.dtype == "f16" else np.float32
    full, _ = run(wl, img, ws)
    for box in boxes:
        win = infer_window(img, ws, box, ndim=wl.ndim, n_in=wl.n_in, channels=wl.channels,
                           factors=wl.factors, steps=wl.steps, fire_rate=wl.fire_rate,
                           seed=wl.seed, dtype=dt)
        sl = tuple(slice(a, b) for a, b in box)
        np.testing.assert_array_equal(win, full[sl])


def test_readout_ties_and_order():
    s = np.zeros((1, 1, 4, 16), np.float32)
    s[0, 0, 0, 14:] = (1.0, 2.0)    # last larger -> 1
    s[0, 0, 1, 14:] = (2.0, 1.0)    # -> 0
    s[0, 0, 2, 14:] = (3.0, 3.0)    # tie -> 0
    s[0, 0, 3, 14:] = (-1.0, -0.5)  # -> 1
    np.testing.assert_array_equal(readout(s)[0, 0], [1, 0, 0, 1])


def test_readout_classes_is_numpy_argmax_of_the_last_k_channels():
    """Without NaNs the K-class readout is numpy's argmax over the last K
    channels (numpy returns the first maximum, i.e. ties go to the lower
    class); values are drawn from a few levels so that ties are frequent."""
    rng = np.random.default_rng(5)
    for k in (2, 3, 5, 13):
        s = rng.integers(-2, 3, size=(2, 7, 9, 16)).astype(np.float32)
        np.testing.assert_array_equal(readout_classes(s, k),
                                      np.argmax(s[..., 16 - k:], axis=-1).astype(np.uint8))


def test_readout_classes_with_two_classes_is_readout():
    rng = np.random.default_rng(6)
    s = rng.integers(-1, 2, size=(1, 11, 13, 16)).astype(np.float32)
    s[0, 0, :3, 15] = np.nan
    s[0, 1, :3, 14] = np.nan
    np.testing.assert_array_equal(readout_classes(s, 2), readout(s))


def test_readout_classes_nan_and_ties_by_hand():
    s = np.zeros((1, 1, 4, 16), np.float32)
    s[0, 0, 0, 13:] = (1.0, np.nan, 2.0)      # NaN skipped, 2.0 wins -> 2
    s[0, 0, 1, 13:] = (np.nan, 5.0, 7.0)      # nothing beats a leading NaN -> 0
    s[0, 0, 2, 13:] = (3.0, 3.0, 3.0)         # three-way tie -> 0
    s[0, 0, 3, 13:] = (-4.0, -1.0, -1.0)      # tie of the two largest -> 1
    np.testing.assert_array_equal(readout_classes(s, 3)[0, 0], [2, 0, 0, 1])


def test_first_level_steps_match_the_papers_bound():
    """With alpha0 = 1 the first level takes max(H, W, D) of its extent, which
    for the paper's pyramids (supplement S7 table, tests/golden) is the finest
    extent's largest side divided by 2 per halving: the max(H, W) / 2^L steps
    of Sec. 3.2 (L counting the halvings)."""
    tasks = json.load(open(os.path.join(GOLDEN, "paper_level_extents.json")))["tasks"]
    for name, t in tasks.items():
        ext = t["extents"]
        halvings = len(ext) - 1
        assert first_level_steps(1.0, ext[-1]) == max(ext[0]) // 2 ** halvings, name
    assert first_level_steps(1.0, tasks["surgery"]["extents"][-1]) == 27


@pytest.mark.parametrize("alpha0,want", [(1.0, 80), (1.5, 120), (2.0, 160)])
def test_first_level_steps_ablation_values(alpha0, want):
    """The ablation's alpha0 values on the prostate volume's coarsest level
    (80 x 80 x 24 after two in-plane halvings of 320 x 320 x 24)."""
    assert first_level_steps(alpha0, (24, 80, 80)) == want


def test_first_level_steps_rounds_down_and_uses_all_axes():
    assert first_level_steps(1.5, (1, 15, 27)) == 40          # 40.5 -> 40
    assert first_level_steps(1.0, (450, 15, 27)) == 450       # time axis counts
    assert first_level_steps(0.0, (3, 4, 5)) == 0


def test_state_magnitude_log_and_tiny_config_finite():
    wl = TINY_2D
    log = InferLog([])
    img = make_image(wl)
    s, seg = infer(img, make_weights(wl), ndim=2, n_in=3, channels=16, factors=wl.factors,
                   steps=wl.steps, fire_rate=0.5, seed=0, dtype=np.float32, log=log)
    assert len(log.max_abs_per_level) == wl.levels
    assert np.isfinite(s).all()
    assert seg.shape == (1, 64, 64) and seg.dtype == np.uint8
