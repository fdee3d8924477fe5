"""Pins of the training-gradient oracle (oracle/train.py) against things other
than itself: central finite differences of the forward in float64 storage,
torch.autograd through an independently written layer-wise PyTorch forward,
the adjoint identity of the upsample, and the fire-rate-0 invariant."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle.octree_nca import nca_step
from oracle.train import LevelGrads

C, H = 16, 64
F64 = np.float64


class W:
    def __init__(self, rng, ndim, scale=0.3):
        taps = 3 ** ndim
        self.conv_w = rng.normal(0, scale, (C, taps))
        self.conv_b = rng.normal(0, scale, (C,))
        self.w1 = rng.normal(0, scale, (H, 2 * C))
        self.b1 = rng.normal(0, scale, (H,))
        self.w2 = rng.normal(0, scale, (C, H))

    def copy(self):
        w = W.__new__(W)
        for k in ("conv_w", "conv_b", "w1", "b1", "w2"):
            setattr(w, k, getattr(self, k).copy())
        return w


KEYS = ("conv_w", "conv_b", "w1", "b1", "w2")


def fd_check(loss, params, grads, rng, n=6, eps=1e-6, rtol=2e-6):
    """Central differences of ``loss`` at ``n`` random entries of each array in
    ``params`` (dict name -> array, perturbed in place) against ``grads``."""
    for name, arr in params.items():
        flat = arr.reshape(-1)
        for i in rng.choice(flat.size, size=min(n, flat.size), replace=False):
            keep = flat[i]
            flat[i] = keep + eps
            lp = loss()
            flat[i] = keep - eps
            lm = loss()
            flat[i] = keep
            num = (lp - lm) / (2 * eps)
            ana = grads[name].reshape(-1)[i]
            assert abs(num - ana) <= rtol * max(1.0, abs(num)), (name, i, num, ana)


@pytest.mark.parametrize("ndim,n_in,shape", [(2, 3, (1, 5, 7)), (3, 1, (3, 4, 5))])
def test_step_vjp_matches_finite_differences(ndim, n_in, shape):
    rng = np.random.default_rng(1)
    w = W(rng, ndim)
    s = rng.normal(0, 1, shape + (C,))
    r = rng.normal(0, 1, shape + (C,))

    def loss():
        out = nca_step(s, w, n_in, ndim, 2, 3, 7, 0.5, F64)
        return float(np.sum(r * out))

    g_in, g = oracle.step_vjp(s, w, n_in, ndim, 2, 3, 7, 0.5, r)
    params = {k: getattr(w, k) for k in KEYS}
    params["state"] = s
    grads = {k: getattr(g, k) for k in KEYS}
    grads["state"] = g_in
    fd_check(loss, params, grads, rng)


def torch_step(s, w, n_in, ndim, mask):
    """Layer-wise PyTorch forward of one step (depthwise conv, concat, two
    linear layers, ReLU, masked residual), written independently of the
    oracle: channels-first tensors for the convolution."""
    c = s.shape[-1]
    if ndim == 2:
        x = s[0].permute(2, 0, 1).unsqueeze(0)                        # [1][C][H][W]
        k = w["conv_w"].reshape(c, 1, 3, 3)
        p = F.conv2d(x, k, w["conv_b"], padding=1, groups=c)[0].permute(1, 2, 0).unsqueeze(0)
    else:
        x = s.permute(3, 0, 1, 2).unsqueeze(0)                        # [1][C][D][H][W]
        k = w["conv_w"].reshape(c, 1, 3, 3, 3)
        p = F.conv3d(x, k, w["conv_b"], padding=1, groups=c)[0].permute(1, 2, 3, 0)
    f = torch.cat([s, p], dim=-1)
    u = F.linear(F.relu(F.linear(f, w["w1"], w["b1"])), w["w2"])
    keep = torch.zeros(c, dtype=s.dtype)
    keep[n_in:] = 1.0
    return s + mask[..., None] * keep * u


@pytest.mark.parametrize("ndim,n_in,shape", [(2, 3, (1, 6, 9)), (3, 1, (4, 5, 6)),
                                             (3, 3, (3, 3, 8))])
def test_step_vjp_matches_torch_autograd(ndim, n_in, shape):
    rng = np.random.default_rng(2)
    w = W(rng, ndim)
    s = rng.normal(0, 1, shape + (C,))
    r = rng.normal(0, 1, shape + (C,))
    mask = oracle.fire_mask(5, 1, 4, shape, 0.5).astype(F64)
    ts = torch.tensor(s, requires_grad=True)
    tw = {k: torch.tensor(getattr(w, k), requires_grad=True) for k in KEYS}
    out = torch_step(ts, tw, n_in, ndim, torch.tensor(mask))
    np.testing.assert_allclose(out.detach().numpy(), nca_step(s, w, n_in, ndim, 1, 4, 5, 0.5, F64),
                               rtol=0, atol=1e-12)
    (out * torch.tensor(r)).sum().backward()
    g_in, g = oracle.step_vjp(s, w, n_in, ndim, 1, 4, 5, 0.5, r)
    np.testing.assert_allclose(g_in, ts.grad.numpy(), rtol=0, atol=1e-10)
    for k in KEYS:
        np.testing.assert_allclose(getattr(g, k), tw[k].grad.numpy(), rtol=0, atol=1e-9,
                                   err_msg=k)


def test_level_vjp_matches_finite_differences():
    rng = np.random.default_rng(3)
    w = W(rng, 2, scale=0.25)
    s0 = rng.normal(0, 1, (1, 6, 6, C))
    r = rng.normal(0, 1, s0.shape)

    def loss():
        st = oracle.level_states(s0, w, 3, 2, 1, 3, 9, 0.5, F64)
        return float(np.sum(r * st[-1]))

    states = oracle.level_states(s0, w, 3, 2, 1, 3, 9, 0.5, F64)
    g_in, g = oracle.level_vjp(states[:-1], w, 3, 2, 1, 9, 0.5, r)
    params = {k: getattr(w, k) for k in KEYS}
    params["state"] = s0
    grads = {k: getattr(g, k) for k in KEYS}
    grads["state"] = g_in
    fd_check(loss, params, grads, rng, n=5)


def test_train_backward_matches_finite_differences():
    """Two levels (8x8 -> 4x4), readout MSE loss, gradients of both levels."""
    rng = np.random.default_rng(4)
    image = rng.uniform(0, 1, (1, 8, 8, 3))
    target = rng.uniform(0, 1, (1, 8, 8, 2))
    ws = [W(rng, 2, scale=0.25), W(rng, 2, scale=0.25)]
    kw = dict(ndim=2, n_in=3, factors=[(1, 2, 2)], seed=11, fire_rate=0.5)

    def loss():
        tape = oracle.train_forward(image, ws, channels=C, steps=[2, 3], dtype=F64, **kw)
        return oracle.readout_mse(tape.final, target)[0]

    tape = oracle.train_forward(image, ws, channels=C, steps=[2, 3], dtype=F64, **kw)
    _, g_final = oracle.readout_mse(tape.final, target)
    grads = oracle.train_backward(tape, ws, g_final=g_final, **kw)
    for lvl in range(2):
        fd_check(loss, {k: getattr(ws[lvl], k) for k in KEYS},
                 {k: getattr(grads[lvl], k) for k in KEYS}, rng, n=4)


def test_upsample_vjp_is_the_adjoint():
    rng = np.random.default_rng(5)
    coarse = rng.normal(0, 1, (2, 3, 4, C))
    fine_img = rng.normal(0, 1, (4, 9, 8, 3))
    y = rng.normal(0, 1, (4, 9, 8, C))
    up = oracle.upsample_inject(coarse, (2, 3, 2), fine_img, F64)
    lhs = np.sum(up[..., 3:] * y[..., 3:])
    rhs = np.sum(coarse * oracle.upsample_vjp(y, (2, 3, 2), 3))
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))
    assert np.all(oracle.upsample_vjp(y, (2, 3, 2), 3)[..., :3] == 0)


def test_fire_rate_zero_gives_no_weight_gradient():
    rng = np.random.default_rng(6)
    w = W(rng, 3)
    s = rng.normal(0, 1, (3, 4, 4, C))
    r = rng.normal(0, 1, s.shape)
    g_in, g = oracle.step_vjp(s, w, 1, 3, 0, 0, 1, 0.0, r)
    np.testing.assert_array_equal(g_in, r)
    for k in KEYS:
        assert np.all(getattr(g, k) == 0), k


def test_readout_mse_gradient():
    rng = np.random.default_rng(7)
    s = rng.normal(0, 1, (1, 3, 4, C))
    y = rng.normal(0, 1, (1, 3, 4, 2))
    loss, g = oracle.readout_mse(s, y)
    assert loss == pytest.approx(0.5 * np.sum((s[..., -2:] - y) ** 2))
    np.testing.assert_array_equal(g[..., :-2], 0)
    np.testing.assert_allclose(g[..., -2:], s[..., -2:] - y)
