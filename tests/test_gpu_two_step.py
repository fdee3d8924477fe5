"""Two steps per launch on large 2D fp32 levels (temporal fusion; legal because
the fire mask is a function of seed, level, step and cell alone).

The two-step row kernel keeps step t's state in LDS and runs step t + 1 on it,
with the same operations in the same order as one launch per step, so its
result must equal the single-step launches bit for bit: checked on ragged
strips (widths around multiples of the 30-cell strip, widths not divisible by
8), short and ragged runs of rows, one- and three-channel images, odd and even
step counts and fire rates 0, 1/2 and 1.  Its parity with the oracle follows
from that and from the single-step kernel's own parity tests (and is also
tested directly by the "mfma_rows" step-kernel cases of the other suites and by
the full-size pathology boxes, where the two-step launches are the default).
The same holds for the ablation's C = 12, H = 48 model (supplement S10), which
runs on the same kernels with channel quad 3 and hidden tile 3 idle."""
import numpy as np
import pytest
import torch

import paper_2508_06993_amd as octnca
from paper_2508_06993_amd.runtime import upload_weights
from synthetic import LevelWeights

pytestmark = pytest.mark.gpu

C, H = 16, 64
SIZES = [(16, 64), (12, 48)]


def rand_weights(rng, scale=0.3, c=C, h=H):
    return LevelWeights(
        conv_w=rng.normal(0, scale, (c, 9)).astype(np.float32),
        conv_b=rng.normal(0, scale, (c,)).astype(np.float32),
        w1=rng.normal(0, scale, (h, 2 * c)).astype(np.float32),
        b1=rng.normal(0, scale, (h,)).astype(np.float32),
        w2=rng.normal(0, scale, (c, h)).astype(np.float32))


def run(kernel, state, w, n_in, steps, rate, level=1, seed=5):
    """run_level with the given step kernel; its result is in buf1 exactly
    when steps is odd (it runs an even number of two-step launches)."""
    b0 = state.clone()
    b1 = torch.full_like(b0, float("nan"))
    c, h = w.w2.shape
    model = octnca.Model(ndim=2, n_in=n_in, kernel=kernel, channels=c, hidden=h)
    which = octnca.octree_nca_run_level(model, b0, b1, upload_weights([w])[0], level, steps,
                                        rate, seed)
    torch.cuda.synchronize()
    return (b1 if which else b0), which


SHAPES = [(1, 1, 1), (1, 2, 29), (1, 3, 30), (1, 5, 31), (1, 9, 59), (1, 33, 61),
          (1, 131, 95), (1, 257, 67), (1, 140, 600)]


@pytest.mark.parametrize("size", SIZES, ids=lambda s: f"c{s[0]}h{s[1]}")
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[1]}x{s[2]}")
@pytest.mark.parametrize("n_in", [1, 3])
def test_two_step_launches_equal_single_steps(gpu, shape, n_in, size):
    c, h = size
    rng = np.random.default_rng(hash((shape, n_in, c)) % 2**32)
    w = rand_weights(rng, c=c, h=h)
    s = torch.from_numpy(rng.normal(0, 1, shape + (c,)).astype(np.float32)).cuda()
    # 4 steps: two two-step launches; 5: two and one single; 7: two and three
    for steps in (1, 4, 5, 7):
        print(f"two-step shape={shape} n_in={n_in} c={c} steps={steps}", flush=True)
        got, which = run("mfma_rows", s, w, n_in, steps, 0.5)
        want, which1 = run("mfma_rows,mfma_1step", s, w, n_in, steps, 0.5)
        assert which1 == steps % 2
        assert which == steps % 2
        assert torch.equal(got, want), (shape, n_in, steps)
        # the input channels are never written
        assert torch.equal(got[..., :n_in], s[..., :n_in])


@pytest.mark.parametrize("size", SIZES, ids=lambda s: f"c{s[0]}h{s[1]}")
@pytest.mark.parametrize("rate", [0.0, 1.0])
def test_two_step_fire_rate_extremes(gpu, rate, size):
    c, h = size
    rng = np.random.default_rng(7)
    w = rand_weights(rng, c=c, h=h)
    s = torch.from_numpy(rng.normal(0, 1, (1, 70, 97, c)).astype(np.float32)).cuda()
    got, _ = run("mfma_rows", s, w, 3, 4, rate)
    want, _ = run("mfma_rows,mfma_1step", s, w, 3, 4, rate)
    assert torch.equal(got, want)
    if rate == 0.0:
        assert torch.equal(got, s)


@pytest.mark.parametrize("size", SIZES, ids=lambda s: f"c{s[0]}h{s[1]}")
def test_two_step_default_on_a_large_level(gpu, size):
    """A level large enough for the default layout to pick the row kernel (and
    with it the two-step launches): 4096 x 1920 cells, strips x runs = 2048.
    Four steps run as two two-step launches, against four single steps."""
    c, h = size
    rng = np.random.default_rng(8)
    w = rand_weights(rng, scale=0.2, c=c, h=h)
    g = torch.Generator(device="cuda").manual_seed(3)
    s = torch.randn((1, 4096, 1920, c), generator=g, device="cuda", dtype=torch.float32)
    model = octnca.Model(ndim=2, n_in=3, channels=c, hidden=h)
    assert octnca.octree_nca_infer_launches(model, (1, 4096, 1920), [], [4]) == [2]
    got, which = run("mfma", s, w, 3, 4, 0.5, level=0)
    want, which1 = run("mfma_1step", s, w, 3, 4, 0.5, level=0)
    assert (which, which1) == (0, 0)
    assert torch.equal(got, want)


@pytest.mark.parametrize("size", SIZES, ids=lambda s: f"c{s[0]}h{s[1]}")
@pytest.mark.parametrize("steps", [(2, 3, 1), (5, 4, 2), (1, 2, 3), (6, 0, 4)],
                         ids=lambda s: "s" + "-".join(map(str, s)))
@pytest.mark.parametrize("factors", [((1, 2, 2), (1, 2, 2)), ((1, 3, 2), (1, 1, 3))],
                         ids=["f22", "f32-13"])
def test_two_step_inference_equals_single_steps(gpu, steps, factors, size):
    """Whole inference with two-step launches (the first of a level fused with
    the upsample when the level has two or more steps) against one step per
    launch: the final state and the readout are equal bit for bit."""
    from synthetic import Workload, make_image, make_weights
    from paper_2508_06993_amd.runtime import Inference, to_device_image
    c, h = size
    wl = Workload(name="two_step_infer", ndim=2, extent=(1, 72, 96), n_in=3, factors=factors,
                  steps=steps, image_kind="uniform", channels=c, hidden=h)
    image = to_device_image(make_image(wl), octnca.Model(ndim=2, n_in=3))
    weights = upload_weights(make_weights(wl))
    out = {}
    for kernel in ("mfma_rows", "mfma_rows,mfma_1step"):
        model = octnca.Model(ndim=2, n_in=3, kernel=kernel, channels=c, hidden=h)
        print(f"two-step inference steps={steps} factors={factors} kernel={kernel}", flush=True)
        run = Inference(model, wl.extent, wl.factors)
        state, seg = run(image, weights, wl.steps, wl.fire_rate, wl.seed)
        torch.cuda.synchronize()
        out[kernel] = (state.clone(), seg.clone())
    assert torch.equal(out["mfma_rows"][0], out["mfma_rows,mfma_1step"][0])
    assert torch.equal(out["mfma_rows"][1], out["mfma_rows,mfma_1step"][1])
