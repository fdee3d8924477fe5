"""Pins for the oracle's image pyramid and state upsampling.

* pooling equals torch's average pooling with kernel = stride = factor;
* on integer-coordinate ramps the block mean has a closed form that is exact in
  float32 (mean of x over a block is f*X + (f-1)/2);
* the pyramid extents for the paper's three tasks equal the supplement S7
  table (tests/golden/paper_level_extents.json);
* nearest upsampling equals torch's nearest interpolation for integer factors
  and maps every fine cell to the parent floor(coordinate / factor).
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pool, build_pyramid, upsample_inject, init_state

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("factor", [(1, 2, 2), (2, 2, 2), (2, 1, 2)])
def test_pool_matches_torch_avg_pool(factor):
    rng = np.random.default_rng(0)
    img = rng.random((4, 6, 10, 3), dtype=np.float32)
    got = pool(img, factor, np.float32)
    x = torch.from_numpy(img.astype(np.float64)).permute(3, 0, 1, 2)[None]   # [1][c][d][h][w]
    want = F.avg_pool3d(x, kernel_size=factor, stride=factor)[0].permute(1, 2, 3, 0).numpy()
    np.testing.assert_array_equal(got, want.astype(np.float32))


def test_pool_2d_matches_avg_pool2d():
    rng = np.random.default_rng(1)
    img = rng.random((1, 12, 8, 3), dtype=np.float32)
    got = pool(img, (1, 2, 2), np.float32)
    x = torch.from_numpy(img[0].astype(np.float64)).permute(2, 0, 1)[None]
    want = F.avg_pool2d(x, 2)[0].permute(1, 2, 0).numpy().astype(np.float32)
    np.testing.assert_array_equal(got[0], want)


def test_pool_exact_on_coordinate_ramps():
    d, h, w = 4, 8, 16
    z, y, x = np.meshgrid(np.arange(d), np.arange(h), np.arange(w), indexing="ij")
    img = np.stack([x, y, z], -1).astype(np.float32)
    pyr = build_pyramid(img, [(2, 2, 2), (1, 2, 2)], np.float32)
    # level 1: mean of x over {2X, 2X+1} = 2X + 0.5
    zz, yy, xx = np.meshgrid(np.arange(2), np.arange(4), np.arange(8), indexing="ij")
    np.testing.assert_array_equal(pyr[1][..., 0], 2 * xx + 0.5)
    np.testing.assert_array_equal(pyr[1][..., 1], 2 * yy + 0.5)
    np.testing.assert_array_equal(pyr[1][..., 2], 2 * zz + 0.5)
    # level 2 = mean over the finest node of 2x4x4 cells: x -> 4X + 1.5, z -> 2Z + 0.5
    zz, yy, xx = np.meshgrid(np.arange(2), np.arange(2), np.arange(4), indexing="ij")
    np.testing.assert_array_equal(pyr[2][..., 0], 4 * xx + 1.5)
    np.testing.assert_array_equal(pyr[2][..., 1], 4 * yy + 1.5)
    np.testing.assert_array_equal(pyr[2][..., 2], 2 * zz + 0.5)


def test_pyramid_is_mean_over_the_finest_node():
    rng = np.random.default_rng(2)
    img = rng.integers(0, 16, size=(4, 8, 8, 2)).astype(np.float32)  # exact sums
    pyr = build_pyramid(img, [(2, 2, 2), (2, 2, 2)], np.float32)
    node = img.reshape(1, 4, 2, 4, 2, 4, 2).mean(axis=(1, 3, 5))
    np.testing.assert_array_equal(pyr[2], node.astype(np.float32))


def test_pool_rejects_indivisible():
    with pytest.raises(ValueError):
        pool(np.zeros((1, 5, 4, 1), np.float32), (1, 2, 2), np.float32)


def _factors_between(extents):
    return [tuple(a // b for a, b in zip(e0, e1)) for e0, e1 in zip(extents, extents[1:])]


@pytest.mark.parametrize("task", ["radiology", "pathology", "surgery"])
def test_pyramid_extents_match_paper_table(task):
    spec = json.load(open(os.path.join(GOLDEN, "paper_level_extents.json")))["tasks"][task]
    ext = [tuple(e) for e in spec["extents"]]
    factors = _factors_between(ext)
    for f in factors:
        assert all(k in (1, 2) for k in f)
    img = np.zeros(ext[0] + (1,), dtype=np.float32)
    pyr = build_pyramid(img, factors, np.float32)
    assert [p.shape[:3] for p in pyr] == ext


@pytest.mark.parametrize("factor", [(1, 2, 2), (2, 2, 2)])
def test_upsample_matches_torch_nearest(factor):
    rng = np.random.default_rng(4)
    coarse = rng.random((2, 3, 5, 16), dtype=np.float32)
    fine_img = rng.random((2 * factor[0], 3 * factor[1], 5 * factor[2], 3), dtype=np.float32)
    got = upsample_inject(coarse, factor, fine_img, np.float32)
    x = torch.from_numpy(coarse).permute(3, 0, 1, 2)[None]
    want = F.interpolate(x, scale_factor=factor, mode="nearest")[0].permute(1, 2, 3, 0).numpy()
    np.testing.assert_array_equal(got[..., 3:], want[..., 3:])
    np.testing.assert_array_equal(got[..., :3], fine_img)


def test_upsample_parent_index_on_coordinates():
    d, h, w = 3, 4, 6
    z, y, x = np.meshgrid(np.arange(d), np.arange(h), np.arange(w), indexing="ij")
    coarse = np.zeros((d, h, w, 16), np.float32)
    coarse[..., 13], coarse[..., 14], coarse[..., 15] = z, y, x
    f = (2, 2, 2)
    fine = upsample_inject(coarse, f, np.zeros((6, 8, 12, 3), np.float32), np.float32)
    zz, yy, xx = np.meshgrid(np.arange(6), np.arange(8), np.arange(12), indexing="ij")
    np.testing.assert_array_equal(fine[..., 13], zz // 2)
    np.testing.assert_array_equal(fine[..., 14], yy // 2)
    np.testing.assert_array_equal(fine[..., 15], xx // 2)


def test_init_state():
    img = np.random.default_rng(5).random((1, 4, 4, 3), dtype=np.float32)
    s = init_state(img, 16, np.float32)
    np.testing.assert_array_equal(s[..., :3], img)
    assert not s[..., 3:].any()


def test_fp16_storage_rounds_once():
    img = np.array([[[[1.0], [2.0 ** -11], [0.0], [0.0]]]], dtype=np.float16)  # 1 x 1 x 4 x 1
    out = pool(img, (1, 1, 2), np.float16)
    # (1 + 2^-11)/2 rounds to nearest even in fp16: 0.5 + 2^-12 is a tie -> 0.5
    assert out.dtype == np.float16
    assert float(out[0, 0, 0, 0]) == 0.5
