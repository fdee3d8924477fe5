"""Pins for the oracle's NCA step (Sec. 3.1; supplement S3, Listing 1).

* perception equals torch's grouped convolution (padding 1) and scipy's
  correlate with a constant-zero border;
* the whole step equals a brute-force per-cell loop written here with plain
  Python floats, and a layer-wise PyTorch pipeline (convolution, concatenation,
  linear, ReLU, linear, mask, add: the "traditional" implementation the paper
  compares its fused kernel against, supplement S4);
* invariants: fire rate 0 and zero second-layer weights give the identity; the
  input channels never change; with zero biases the step is positively
  homogeneous of degree 1; away from the border it is translation
  equivariant when every cell fires.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.ndimage import correlate

from oracle import perceive, nca_step, tap_offsets, fire_mask
from synthetic import LevelWeights

from brute import brute_step

C, H = 16, 64


def rand_weights(rng, ndim, scale=0.1):
    taps = 3 ** ndim
    return LevelWeights(
        conv_w=rng.normal(0, scale, (C, taps)).astype(np.float32),
        conv_b=rng.normal(0, scale, (C,)).astype(np.float32),
        w1=rng.normal(0, scale, (H, 2 * C)).astype(np.float32),
        b1=rng.normal(0, scale, (H,)).astype(np.float32),
        w2=rng.normal(0, scale, (C, H)).astype(np.float32))


def rand_state(rng, shape):
    return rng.normal(0, 1, shape + (C,)).astype(np.float32)


@pytest.mark.parametrize("ndim,shape", [(2, (1, 7, 9)), (3, (4, 5, 6))])
def test_perceive_matches_torch_grouped_conv(ndim, shape):
    rng = np.random.default_rng(0)
    w = rand_weights(rng, ndim)
    s = rand_state(rng, shape).astype(np.float64)
    got = perceive(s, w.conv_w, w.conv_b, ndim)
    wt = torch.from_numpy(w.conv_w.astype(np.float64))
    bt = torch.from_numpy(w.conv_b.astype(np.float64))
    if ndim == 2:
        x = torch.from_numpy(s[0]).permute(2, 0, 1)[None]
        y = F.conv2d(x, wt.reshape(C, 1, 3, 3), bt, padding=1, groups=C)
        want = y[0].permute(1, 2, 0).numpy()[None]
    else:
        x = torch.from_numpy(s).permute(3, 0, 1, 2)[None]
        y = F.conv3d(x, wt.reshape(C, 1, 3, 3, 3), bt, padding=1, groups=C)
        want = y[0].permute(1, 2, 3, 0).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_perceive_matches_scipy_correlate():
    rng = np.random.default_rng(1)
    w = rand_weights(rng, 3)
    s = rand_state(rng, (3, 4, 5)).astype(np.float64)
    got = perceive(s, w.conv_w, w.conv_b, 3)
    for c in range(C):
        k = w.conv_w[c].astype(np.float64).reshape(3, 3, 3)
        want = correlate(s[..., c], k, mode="constant", cval=0.0) + w.conv_b[c]
        np.testing.assert_allclose(got[..., c], want, rtol=1e-12, atol=1e-12)


def test_tap_order():
    assert tap_offsets(2)[0] == (0, -1, -1) and tap_offsets(2)[5] == (0, 0, 1)
    assert tap_offsets(3)[0] == (-1, -1, -1) and tap_offsets(3)[13] == (0, 0, 0)
    assert len(tap_offsets(3)) == 27


@pytest.mark.parametrize("ndim,shape,n_in", [(2, (1, 5, 6), 3), (3, (3, 4, 3), 1), (3, (2, 3, 5), 3)])
def test_step_matches_brute_force(ndim, shape, n_in):
    rng = np.random.default_rng(2)
    w = rand_weights(rng, ndim)
    s = rand_state(rng, shape)
    got = nca_step(s, w, n_in, ndim, level=1, step=3, seed=5, fire_rate=0.5, dtype=np.float32)
    want = brute_step(s, w, n_in, ndim, 1, 3, 5, 0.5)
    np.testing.assert_allclose(got, want, rtol=2e-7, atol=1e-7)


@pytest.mark.parametrize("c,h,ndim,n_in", [(12, 48, 2, 3), (20, 100, 3, 1), (12, 48, 3, 3)])
def test_step_matches_brute_force_other_model_sizes(c, h, ndim, n_in):
    """The ablation's model sizes C/H = 12/48 and 20/100 (supplement S10)."""
    rng = np.random.default_rng(8)
    taps = 3 ** ndim
    w = LevelWeights(conv_w=rng.normal(0, 0.1, (c, taps)).astype(np.float32),
                     conv_b=rng.normal(0, 0.1, (c,)).astype(np.float32),
                     w1=rng.normal(0, 0.1, (h, 2 * c)).astype(np.float32),
                     b1=rng.normal(0, 0.1, (h,)).astype(np.float32),
                     w2=rng.normal(0, 0.1, (c, h)).astype(np.float32))
    s = rng.normal(0, 1, (2, 4, 5, c) if ndim == 3 else (1, 5, 6, c)).astype(np.float32)
    got = nca_step(s, w, n_in, ndim, level=0, step=1, seed=2, fire_rate=0.5, dtype=np.float32)
    want = brute_step(s, w, n_in, ndim, 0, 1, 2, 0.5)
    np.testing.assert_allclose(got, want, rtol=2e-7, atol=1e-7)


def layerwise_step(state, w, n_in, ndim, level, t, seed, fire_rate):
    """The layer-wise PyTorch pipeline, float64 on the CPU."""
    s = torch.from_numpy(state.astype(np.float64))
    if ndim == 2:
        x = s[0].permute(2, 0, 1)[None]
        conv = F.conv2d(x, torch.from_numpy(w.conv_w.astype(np.float64)).reshape(C, 1, 3, 3),
                        torch.from_numpy(w.conv_b.astype(np.float64)), padding=1, groups=C)
        conv = conv[0].permute(1, 2, 0)[None]
    else:
        x = s.permute(3, 0, 1, 2)[None]
        conv = F.conv3d(x, torch.from_numpy(w.conv_w.astype(np.float64)).reshape(C, 1, 3, 3, 3),
                        torch.from_numpy(w.conv_b.astype(np.float64)), padding=1, groups=C)
        conv = conv[0].permute(1, 2, 3, 0)
    feat = torch.cat([s, conv], dim=-1)
    hid = F.relu(F.linear(feat, torch.from_numpy(w.w1.astype(np.float64)),
                          torch.from_numpy(w.b1.astype(np.float64))))
    upd = F.linear(hid, torch.from_numpy(w.w2[n_in:].astype(np.float64)))
    m = torch.from_numpy(fire_mask(seed, level, t, state.shape[:3], fire_rate).astype(np.float64))
    new_hidden = s[..., n_in:] + m[..., None] * upd
    return torch.cat([s[..., :n_in], new_hidden], dim=-1).numpy().astype(np.float32)


@pytest.mark.parametrize("ndim,shape,n_in", [(2, (1, 33, 47), 3), (3, (6, 9, 11), 1), (3, (5, 8, 7), 3)])
def test_step_matches_layerwise_pipeline(ndim, shape, n_in):
    rng = np.random.default_rng(3)
    w = rand_weights(rng, ndim)
    s = rand_state(rng, shape)
    got = nca_step(s, w, n_in, ndim, level=0, step=7, seed=1, fire_rate=0.5, dtype=np.float32)
    want = layerwise_step(s, w, n_in, ndim, 0, 7, 1, 0.5)
    np.testing.assert_allclose(got, want, rtol=2e-7, atol=1e-7)


@pytest.mark.parametrize("ndim", [2, 3])
def test_fire_rate_zero_is_identity(ndim):
    rng = np.random.default_rng(4)
    w = rand_weights(rng, ndim)
    s = rand_state(rng, (1, 8, 8) if ndim == 2 else (4, 5, 6))
    out = nca_step(s, w, 3, ndim, 0, 0, 0, 0.0, np.float32)
    np.testing.assert_array_equal(out, s)


def test_zero_second_layer_is_identity():
    rng = np.random.default_rng(5)
    w = rand_weights(rng, 2)
    w.w2[:] = 0
    s = rand_state(rng, (1, 9, 7))
    np.testing.assert_array_equal(nca_step(s, w, 3, 2, 0, 0, 0, 1.0, np.float32), s)


def test_all_zero_weights_is_identity():
    rng = np.random.default_rng(6)
    w = rand_weights(rng, 3, scale=0.0)
    s = rand_state(rng, (3, 4, 5))
    np.testing.assert_array_equal(nca_step(s, w, 1, 3, 0, 0, 0, 1.0, np.float32), s)


@pytest.mark.parametrize("n_in", [1, 3])
def test_input_channels_unchanged(n_in):
    rng = np.random.default_rng(7)
    w = rand_weights(rng, 2, scale=1.0)
    s = rand_state(rng, (1, 12, 10))
    out = s
    for t in range(5):
        out = nca_step(out, w, n_in, 2, 0, t, 0, 1.0, np.float32)
    np.testing.assert_array_equal(out[..., :n_in], s[..., :n_in])
    assert np.abs(out[..., n_in:] - s[..., n_in:]).max() > 0


def test_positive_homogeneity_without_biases():
    rng = np.random.default_rng(8)
    w = rand_weights(rng, 2)
    w.conv_b[:] = 0
    w.b1[:] = 0
    s = rand_state(rng, (1, 10, 10))
    a = nca_step(s, w, 3, 2, 0, 0, 0, 0.5, np.float32)
    b = nca_step(2 * s, w, 3, 2, 0, 0, 0, 0.5, np.float32)
    np.testing.assert_array_equal(b, 2 * a)


def test_translation_equivariance_when_all_fire():
    rng = np.random.default_rng(9)
    w = rand_weights(rng, 2)
    s = rand_state(rng, (1, 20, 20))
    shifted = np.roll(s, (3, -2), axis=(1, 2))
    a = nca_step(s, w, 3, 2, 0, 0, 0, 1.0, np.float32)
    b = nca_step(shifted, w, 3, 2, 0, 0, 0, 1.0, np.float32)
    # compare cells whose neighbourhood did not touch the border or the wrap
    np.testing.assert_array_equal(np.roll(a, (3, -2), axis=(1, 2))[:, 5:16, 2:16],
                                  b[:, 5:16, 2:16])


def test_fire_mask_gates_whole_cell():
    rng = np.random.default_rng(10)
    w = rand_weights(rng, 2)
    s = rand_state(rng, (1, 16, 16))
    out = nca_step(s, w, 3, 2, 2, 4, 3, 0.5, np.float32)
    m = fire_mask(3, 2, 4, (1, 16, 16), 0.5)
    changed = (out != s).any(axis=-1)
    assert not changed[~m].any()
    assert changed[m].all()


def test_fp16_state_stays_fp16():
    rng = np.random.default_rng(11)
    w = rand_weights(rng, 3)
    s = rand_state(rng, (2, 4, 4)).astype(np.float16)
    out = nca_step(s, w, 3, 3, 0, 0, 0, 1.0, np.float16)
    assert out.dtype == np.float16
    ref = layerwise_step(s.astype(np.float32), w, 3, 3, 0, 0, 0, 1.0)
    # one rounding to fp16 from (nearly) the same float64 value: within one fp16 ulp
    ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float32)
    assert (np.abs(out.astype(np.float32) - ref) <= ulp).all()
