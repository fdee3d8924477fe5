"""GPU parity of the training-gradient entry points against the oracle
(oracle/train.py), through the C ABI: the backward of one step (state
gradient and the five weight gradients), its accumulation and in-place use,
the upsample's adjoint, the readout MSE, and the whole fused training step.

Bounds (max |g - o| / max |o|): the GPU computes in fp32 what the oracle
computes in fp64 from the same fp32 inputs.  A state gradient is a sum of a
few dozen fp32 products per cell: 2e-5.  A weight gradient sums one product
per cell over every cell (fp32 within chunks of 32 cells, fp64 across
chunks): 1e-4.  The training step also differs in its forward states (the
matrix-core MLP with split-bf16 operands, products to about 2^-16, against
the oracle's fp64 arithmetic rounded to fp32 per step), which the steps
carry along: 1e-3."""
import numpy as np
import pytest
import torch

import oracle
import paper_2508_06993_amd as octnca
from paper_2508_06993_amd.runtime import upload_weights
from synthetic import LevelWeights

from parity import to_np, max_rel_err

pytestmark = pytest.mark.gpu

C, H = 16, 64
KEYS = ("conv_w", "conv_b", "w1", "b1", "w2")
TOL_STATE, TOL_WEIGHT, TOL_TRAIN = 2e-5, 1e-4, 1e-3


def rand_weights(rng, ndim, scale=0.3, c=C, h=H):
    taps = 3 ** ndim
    return LevelWeights(
        conv_w=rng.normal(0, scale, (c, taps)).astype(np.float32),
        conv_b=rng.normal(0, scale, (c,)).astype(np.float32),
        w1=rng.normal(0, scale, (h, 2 * c)).astype(np.float32),
        b1=rng.normal(0, scale, (h,)).astype(np.float32),
        w2=rng.normal(0, scale, (c, h)).astype(np.float32))


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def zero_grads(w):
    return {k: torch.zeros(getattr(w, k).shape, dtype=torch.float32, device="cuda") for k in KEYS}


def step_backward_gpu(model, state, g_out, w, level, step, rate, seed, grads=None,
                      in_place=False):
    s, g = dev(state), dev(g_out)
    gin = g if in_place else torch.empty_like(g)
    grads = zero_grads(w) if grads is None else grads
    ws = torch.empty(octnca.octree_nca_step_backward_workspace_bytes(model, state.shape[:3]),
                     dtype=torch.uint8, device="cuda")
    octnca.octree_nca_step_backward(model, s, g, upload_weights([w])[0], level, step, rate, seed,
                                    gin, grads, ws)
    torch.cuda.synchronize()
    return to_np(gin), {k: to_np(v) for k, v in grads.items()}, grads


STEP_CASES = [(2, 3, (1, 20, 70)), (2, 1, (1, 9, 33)), (2, 3, (1, 64, 96)),
              (3, 1, (5, 9, 10)), (3, 3, (6, 17, 9)), (2, 3, (1, 1, 1))]


@pytest.mark.parametrize("ndim,n_in,shape", STEP_CASES)
def test_step_backward_matches_oracle(gpu, ndim, n_in, shape):
    rng = np.random.default_rng(31)
    w = rand_weights(rng, ndim)
    s = rng.normal(0, 1, shape + (C,)).astype(np.float32)
    g_out = rng.normal(0, 1, shape + (C,)).astype(np.float32)
    model = octnca.Model(ndim=ndim, n_in=n_in)
    gin, grads, _ = step_backward_gpu(model, s, g_out, w, 2, 5, 0.5, 9)
    want_in, want = oracle.step_vjp(s, w, n_in, ndim, 2, 5, 9, 0.5, g_out)
    assert max_rel_err(gin, want_in) <= TOL_STATE
    for k in KEYS:
        assert max_rel_err(grads[k], getattr(want, k)) <= TOL_WEIGHT, k
    assert np.all(grads["w2"][:n_in] == 0)


def test_step_backward_in_place_and_accumulating(gpu):
    rng = np.random.default_rng(32)
    w = rand_weights(rng, 3)
    s = rng.normal(0, 1, (4, 10, 12, C)).astype(np.float32)
    g_out = rng.normal(0, 1, s.shape).astype(np.float32)
    model = octnca.Model(ndim=3, n_in=1)
    gin_a, grads_a, acc = step_backward_gpu(model, s, g_out, w, 1, 2, 0.5, 4)
    gin_b, grads_b, _ = step_backward_gpu(model, s, g_out, w, 1, 2, 0.5, 4, in_place=True)
    np.testing.assert_array_equal(gin_a, gin_b)
    for k in KEYS:
        np.testing.assert_array_equal(grads_a[k], grads_b[k])
    # a second call adds to the same gradients
    _, grads_2, _ = step_backward_gpu(model, s, g_out, w, 1, 2, 0.5, 4, grads=acc)
    for k in KEYS:
        np.testing.assert_allclose(grads_2[k], 2 * grads_a[k], rtol=1e-6, atol=1e-6, err_msg=k)


def test_step_backward_fire_rate_zero(gpu):
    rng = np.random.default_rng(33)
    w = rand_weights(rng, 2)
    s = rng.normal(0, 1, (1, 12, 40, C)).astype(np.float32)
    g_out = rng.normal(0, 1, s.shape).astype(np.float32)
    gin, grads, _ = step_backward_gpu(octnca.Model(ndim=2, n_in=3), s, g_out, w, 0, 0, 0.0, 1)
    np.testing.assert_array_equal(gin, g_out)
    for k in KEYS:
        assert np.all(grads[k] == 0), k


@pytest.mark.parametrize("c,h,ndim", [(12, 48, 2), (20, 100, 3)])
def test_step_backward_other_model_sizes(gpu, c, h, ndim):
    rng = np.random.default_rng(34)
    w = rand_weights(rng, ndim, c=c, h=h)
    shape = (1, 11, 37) if ndim == 2 else (3, 7, 9)
    s = rng.normal(0, 1, shape + (c,)).astype(np.float32)
    g_out = rng.normal(0, 1, s.shape).astype(np.float32)
    model = octnca.Model(ndim=ndim, n_in=3, channels=c, hidden=h)
    gin, grads, _ = step_backward_gpu(model, s, g_out, w, 1, 3, 0.5, 2)
    want_in, want = oracle.step_vjp(s, w, 3, ndim, 1, 3, 2, 0.5, g_out)
    assert max_rel_err(gin, want_in) <= TOL_STATE
    for k in KEYS:
        assert max_rel_err(grads[k], getattr(want, k)) <= TOL_WEIGHT, k


@pytest.mark.parametrize("ndim,coarse,factor", [(2, (1, 5, 7), (1, 2, 2)),
                                                (3, (3, 4, 5), (2, 2, 2)),
                                                (3, (2, 3, 4), (1, 3, 2))])
def test_upsample_backward_matches_oracle(gpu, ndim, coarse, factor):
    rng = np.random.default_rng(35)
    fine = tuple(a * f for a, f in zip(coarse, factor))
    g_fine = rng.normal(0, 1, fine + (C,)).astype(np.float32)
    g_coarse = torch.empty(coarse + (C,), dtype=torch.float32, device="cuda")
    octnca.octree_nca_upsample_backward(octnca.Model(ndim=ndim, n_in=3), dev(g_fine), factor,
                                        g_coarse)
    torch.cuda.synchronize()
    want = oracle.upsample_vjp(g_fine, factor, 3)
    assert max_rel_err(to_np(g_coarse), want) <= 1e-6
    assert np.all(to_np(g_coarse)[..., :3] == 0)


def test_readout_mse_matches_oracle(gpu):
    rng = np.random.default_rng(36)
    s = rng.normal(0, 1, (1, 33, 65, C)).astype(np.float32)
    y = rng.uniform(0, 1, (1, 33, 65, 2)).astype(np.float32)
    model = octnca.Model(ndim=2, n_in=3)
    grad = torch.empty(s.shape, dtype=torch.float32, device="cuda")
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    ws = torch.empty(octnca.octree_nca_readout_mse_workspace_bytes(s.shape[:3]),
                     dtype=torch.uint8, device="cuda")
    octnca.octree_nca_readout_mse(model, dev(s), dev(y), grad, loss, ws)
    torch.cuda.synchronize()
    want_loss, want_grad = oracle.readout_mse(s, y)
    assert float(to_np(loss)[0]) == pytest.approx(want_loss, rel=1e-12)
    np.testing.assert_array_equal(to_np(grad), want_grad.astype(np.float32))


TRAIN_CASES = [
    ("2d-3lvl", 2, 3, (1, 32, 48), ((1, 2, 2), (1, 2, 2)), (3, 2, 4)),
    ("3d-2lvl", 3, 1, (4, 16, 24), ((2, 2, 2),), (2, 3)),
    ("2dt-2lvl", 3, 3, (6, 8, 20), ((1, 2, 2),), (3, 1)),
    # a level without steps between two with several (its gradient passes
    # straight to the upsample's adjoint); ragged backward tiles
    ("2d-zero-steps", 2, 3, (1, 36, 68), ((1, 2, 2), (1, 3, 2)), (4, 0, 3)),
    ("2d-5steps", 2, 1, (1, 70, 40), ((1, 2, 2),), (5, 2)),
]


@pytest.mark.parametrize("name,ndim,n_in,extent,factors,steps", TRAIN_CASES,
                         ids=[c[0] for c in TRAIN_CASES])
def test_train_step_matches_oracle(gpu, name, ndim, n_in, extent, factors, steps):
    rng = np.random.default_rng(37)
    levels = len(steps)
    image = rng.uniform(0, 1, extent + (n_in,)).astype(np.float32)
    target = rng.uniform(0, 1, extent + (2,)).astype(np.float32)
    ws_list = [rand_weights(rng, ndim, scale=0.2) for _ in range(levels)]
    model = octnca.Model(ndim=ndim, n_in=n_in)
    grads = [zero_grads(w) for w in ws_list]
    for g in grads:                       # overwritten, not accumulated
        for t in g.values():
            t.fill_(7.0)
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    final = torch.empty(extent + (C,), dtype=torch.float32, device="cuda")
    work = torch.empty(octnca.octree_nca_train_workspace_bytes(model, extent, factors, steps),
                       dtype=torch.uint8, device="cuda")
    octnca.octree_nca_train_step(model, dev(image), factors, upload_weights(ws_list), steps, 0.5,
                                 3, dev(target), work, grads, loss, final)
    torch.cuda.synchronize()
    kw = dict(ndim=ndim, n_in=n_in, factors=factors, seed=3, fire_rate=0.5)
    tape = oracle.train_forward(image, ws_list, channels=C, steps=steps, dtype=np.float32, **kw)
    want_loss, g_final = oracle.readout_mse(tape.final, target)
    want = oracle.train_backward(tape, ws_list, g_final=g_final, **kw)
    assert max_rel_err(to_np(final), tape.final) <= TOL_TRAIN
    assert float(to_np(loss)[0]) == pytest.approx(want_loss, rel=TOL_TRAIN)
    for lvl in range(levels):
        for k in KEYS:
            err = max_rel_err(to_np(grads[lvl][k]), getattr(want[lvl], k))
            assert err <= TOL_TRAIN, (lvl, k, err)
