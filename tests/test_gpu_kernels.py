"""GPU parity of the individual entry points against the oracle, through the
C ABI: fire masks and upsampling bit-exact, pyramid values within rounding of
the fp64 mean (exact on integer ramps), one NCA step and a level's steps
within the storage type's bound, plus the step's invariants on the GPU."""
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
NP_DT = {"f32": np.float32, "f16": np.float16}
T_DT = {"f32": torch.float32, "f16": torch.float16}


def rand_weights(rng, ndim, scale=0.1, c=C, h=H):
    taps = 3 ** ndim
    return LevelWeights(
        conv_w=rng.normal(0, scale, (c, taps)).astype(np.float32),
        conv_b=rng.normal(0, scale, (c,)).astype(np.float32),
        w1=rng.normal(0, scale, (h, 2 * c)).astype(np.float32),
        b1=rng.normal(0, scale, (h,)).astype(np.float32),
        w2=rng.normal(0, scale, (c, h)).astype(np.float32))


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


# ---------------------------------------------------------------------------
# fire mask: bit-exact
# ---------------------------------------------------------------------------

MASK_CASES = [
    ((1, 1, 1), 0, 0, 0, 0.5), ((1, 7, 9), 0, 3, 1, 0.5), ((3, 5, 6), 12345, 2, 19, 0.5),
    ((1, 64, 64), 0, 0, 0, 0.5), ((1, 33, 257), 2 ** 63 + 5, 5, 7, 0.3),
    ((1, 16, 16), 9, 1, 2, 0.0), ((1, 16, 16), 9, 1, 2, 1.0), ((4, 9, 11), 77, 4, 15, 0.999),
    ((2, 100, 1000), 3, 0, 11, 0.5),
]


@pytest.mark.parametrize("extent,seed,level,step,rate", MASK_CASES)
def test_fire_mask_bit_exact(gpu, extent, seed, level, step, rate):
    mask = torch.empty(extent, dtype=torch.uint8, device=gpu)
    octnca.octree_nca_fire_mask(seed, level, step, extent, rate, mask)
    torch.cuda.synchronize()
    want = oracle.fire_mask(seed, level, step, extent, rate).astype(np.uint8)
    np.testing.assert_array_equal(to_np(mask), want)


# ---------------------------------------------------------------------------
# pyramid
# ---------------------------------------------------------------------------

POOL_CASES = [("f32", 2, (1, 64, 96), [(1, 2, 2)] * 3, 3), ("f32", 3, (8, 24, 20),
              [(2, 2, 2), (1, 2, 2)], 1), ("f16", 3, (8, 24, 20), [(2, 2, 2), (2, 2, 1)], 3),
              ("f16", 2, (1, 40, 36), [(1, 2, 2), (1, 2, 3)], 3), ("f32", 3, (6, 9, 4),
              [(3, 3, 4)], 3), ("f16", 3, (4, 20, 36), [(1, 2, 2), (2, 2, 2)], 1),
              ("f32", 2, (1, 34, 18), [(1, 2, 2)], 1)]


@pytest.mark.parametrize("dt,ndim,extent,factors,n_in", POOL_CASES)
def test_pyramid_matches_oracle(gpu, dt, ndim, extent, factors, n_in):
    rng = np.random.default_rng(5)
    img = rng.random(extent + (n_in,), dtype=np.float32).astype(NP_DT[dt])
    model = octnca.Model(ndim=ndim, n_in=n_in, dtype=dt)
    want = oracle.build_pyramid(img, factors, NP_DT[dt])
    outs = [torch.empty(w.shape, dtype=T_DT[dt], device=gpu) for w in want[1:]]
    octnca.octree_nca_build_pyramid(model, dev(img), factors, outs)
    torch.cuda.synchronize()
    for lvl, (g, w) in enumerate(zip(outs, want[1:]), start=1):
        g = to_np(g).astype(np.float64)
        w = w.astype(np.float64)
        if dt == "f32":
            np.testing.assert_allclose(g, w, rtol=1e-6, atol=1e-7, err_msg=f"level {lvl}")
        else:   # one fp16 rounding of an fp32 sum vs of an fp64 sum
            np.testing.assert_allclose(g, w, rtol=1e-3, atol=1e-4, err_msg=f"level {lvl}")


def test_pyramid_exact_on_coordinate_ramps(gpu):
    """Channel k holds coordinate k of each cell; each pooled value must be the
    exact block mean f*X + (f-1)/2 (all values are small dyadic numbers)."""
    d, h, w = 8, 32, 48
    z, y, x = np.meshgrid(np.arange(d), np.arange(h), np.arange(w), indexing="ij")
    img = np.stack([x, y, z], -1).astype(np.float32)
    factors = [(2, 2, 2), (1, 2, 2), (2, 2, 1)]
    model = octnca.Model(ndim=3, n_in=3)
    want = oracle.build_pyramid(img, factors, np.float32)
    outs = [torch.empty(t.shape, dtype=torch.float32, device=gpu) for t in want[1:]]
    octnca.octree_nca_build_pyramid(model, dev(img), factors, outs)
    torch.cuda.synchronize()
    cum = np.array([1, 1, 1])
    for g, wt, f in zip(outs, want[1:], factors):
        cum = cum * np.array(f)
        zz, yy, xx = np.meshgrid(*(np.arange(n) for n in wt.shape[:3]), indexing="ij")
        exact = np.stack([cum[2] * xx + (cum[2] - 1) / 2, cum[1] * yy + (cum[1] - 1) / 2,
                          cum[0] * zz + (cum[0] - 1) / 2], -1)
        np.testing.assert_array_equal(to_np(g), exact.astype(np.float32))
        np.testing.assert_array_equal(to_np(g), wt)


# ---------------------------------------------------------------------------
# upsample + inject: bit-exact
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt,ndim,coarse,factor,n_in",
                         [("f32", 2, (1, 5, 7), (1, 2, 2), 3), ("f16", 3, (3, 4, 5), (2, 2, 2), 3),
                          ("f32", 3, (2, 3, 3), (1, 2, 2), 1), ("f16", 2, (1, 9, 4), (1, 3, 2), 1),
                          ("f32", 3, (1, 1, 1), (4, 4, 4), 3)])
def test_upsample_bit_exact(gpu, dt, ndim, coarse, factor, n_in):
    rng = np.random.default_rng(7)
    cs = rng.normal(0, 1, coarse + (C,)).astype(NP_DT[dt])
    fine_ext = tuple(a * b for a, b in zip(coarse, factor))
    img = rng.random(fine_ext + (n_in,), dtype=np.float32).astype(NP_DT[dt])
    model = octnca.Model(ndim=ndim, n_in=n_in, dtype=dt)
    out = torch.full(fine_ext + (C,), 99.0, dtype=T_DT[dt], device=gpu)
    octnca.octree_nca_upsample(model, dev(cs), factor, dev(img), out)
    torch.cuda.synchronize()
    want = oracle.upsample_inject(cs, factor, img, NP_DT[dt])
    np.testing.assert_array_equal(to_np(out), want)


def test_upsample_parent_indices_on_coordinates(gpu):
    """Hidden channels hold the coarse cell's coordinates as exact floats."""
    cd, ch, cw = 3, 5, 6
    f = (2, 2, 2)
    cs = np.zeros((cd, ch, cw, C), np.float32)
    z, y, x = np.meshgrid(np.arange(cd), np.arange(ch), np.arange(cw), indexing="ij")
    cs[..., 3], cs[..., 4], cs[..., 5] = x, y, z
    fine = (cd * 2, ch * 2, cw * 2)
    img = np.zeros(fine + (3,), np.float32)
    out = torch.empty(fine + (C,), dtype=torch.float32, device=gpu)
    octnca.octree_nca_upsample(octnca.Model(ndim=3, n_in=3), dev(cs), f, dev(img), out)
    torch.cuda.synchronize()
    o = to_np(out)
    fz, fy, fx = np.meshgrid(*(np.arange(n) for n in fine), indexing="ij")
    np.testing.assert_array_equal(o[..., 3], fx // 2)
    np.testing.assert_array_equal(o[..., 4], fy // 2)
    np.testing.assert_array_equal(o[..., 5], fz // 2)


def test_readout_matches_oracle(gpu):
    rng = np.random.default_rng(3)
    s = rng.normal(0, 1, (2, 17, 31, C)).astype(np.float32)
    s[0, 0, :5, 14] = s[0, 0, :5, 15]      # ties -> 0
    seg = torch.empty((2, 17, 31), dtype=torch.uint8, device=gpu)
    octnca.octree_nca_readout(octnca.Model(ndim=3, n_in=1), dev(s), seg)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(seg), oracle.readout(s))


@pytest.mark.parametrize("dt,classes,n_in", [("f32", 2, 3), ("f32", 5, 3), ("f32", 13, 3),
                                              ("f16", 4, 1), ("f16", 15, 1)])
def test_readout_classes_matches_oracle(gpu, dt, classes, n_in):
    """Bit-exact against the oracle: values drawn from a few levels (frequent
    ties), some NaNs, both storage types."""
    rng = np.random.default_rng(4 + classes)
    s = rng.integers(-3, 4, size=(3, 13, 29, C)).astype(NP_DT[dt])
    s[0, 1, :7, C - classes] = np.nan
    s[1, 2, :5, C - 1] = np.nan
    seg = torch.empty((3, 13, 29), dtype=torch.uint8, device=gpu)
    octnca.octree_nca_readout_classes(octnca.Model(ndim=3, n_in=n_in, dtype=dt), dev(s),
                                      classes, seg)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(seg), oracle.readout_classes(s, classes))
    if classes == 2:
        np.testing.assert_array_equal(to_np(seg), oracle.readout(s))


# ---------------------------------------------------------------------------
# one step / one level
# ---------------------------------------------------------------------------

STEP_CASES = [
    ("f32", 2, 3, (1, 37, 83)), ("f32", 2, 1, (1, 8, 32)), ("f32", 2, 3, (1, 1, 1)),
    ("f32", 2, 3, (1, 1, 70)), ("f32", 3, 1, (7, 19, 13)), ("f32", 3, 3, (5, 9, 17)),
    ("f32", 3, 1, (1, 1, 1)), ("f16", 2, 3, (1, 21, 45)), ("f16", 3, 3, (6, 11, 10)),
    ("f16", 3, 1, (3, 8, 8)),
    # several 32-plane z runs with a ragged last run, ragged y tiles, 8-aligned
    # and unaligned rows
    ("f32", 3, 1, (70, 12, 40)), ("f16", 3, 3, (70, 10, 36)), ("f16", 3, 3, (33, 16, 64)),
    # several 64-row runs of the 2D row layout with ragged last runs and strips
    ("f32", 2, 3, (1, 150, 70)), ("f16", 2, 3, (1, 131, 40)),
]


# Max relative error bounds (max |g - o| / max |o|) after one step and after
# nine steps of one level, per storage type and step kernel.  fp32 operands
# (vector FMAs or fp32 MFMA) differ from the fp64 oracle by fp32 rounding only;
# split-bf16 operands keep products to about 2^-16 relative; with fp16 states
# the storage rounding (2^-11) dominates, plus fp16 MLP operands and (3D)
# fp16 perception sums on "mfma".
# (one step, nine steps) bounds on max |g - o| / max |o|.  fp32 operands:
# rounding only.  Split bf16 (x3): products to ~2^-16.  The default MLP for
# fp32 states (scaled fp16 activations, split fp16 weights): every feature and
# hidden unit rounded to fp16 (2^-12 relative), which gives ~1e-4 on one step
# of these N(0, 1) states; the nine-step bound stays below the 1e-3 bound of a
# whole inference.  fp16 states: storage rounding (2^-11) dominates.
STEP_TOL = {
    ("f32", "valu"): (2e-6, 1e-4), ("f32", "mfma_f32"): (2e-6, 1e-4),
    ("f32", "mfma_bf16x3"): (5e-5, 5e-4),
    ("f32", "mfma"): (3e-4, 5e-4), ("f32", "mfma_rows"): (3e-4, 5e-4),
    ("f32", "mfma_tiles"): (3e-4, 5e-4), ("f32", "mfma_1step"): (3e-4, 5e-4),
    ("f16", "valu"): (1e-3, 1e-2), ("f16", "mfma_f32"): (1e-3, 1e-2),
    ("f16", "mfma_bf16x3"): (1e-3, 1e-2),
    ("f16", "mfma"): (3e-3, 1e-2), ("f16", "mfma_rows"): (3e-3, 1e-2),
    ("f16", "mfma_tiles"): (3e-3, 1e-2), ("f16", "mfma_1step"): (3e-3, 1e-2),
}


def run_level_gpu(model, state, w, level, steps, rate, seed):
    b0 = dev(state)
    b1 = torch.empty_like(b0)
    which = octnca.octree_nca_run_level(model, b0, b1, upload_weights([w])[0], level, steps, rate,
                                        seed)
    torch.cuda.synchronize()
    return to_np(b1 if which else b0), which


@pytest.mark.parametrize("dt,ndim,n_in,shape", STEP_CASES)
def test_one_step_matches_oracle(gpu, step_kernel, dt, ndim, n_in, shape):
    rng = np.random.default_rng(11)
    w = rand_weights(rng, ndim)
    s = rng.normal(0, 1, shape + (C,)).astype(NP_DT[dt])
    got, which = run_level_gpu(octnca.Model(ndim=ndim, n_in=n_in, dtype=dt, kernel=step_kernel),
                               s, w, 2, 1, 0.5, 42)
    assert which == 1
    want = oracle.nca_step(s, w, n_in, ndim, 2, 0, 42, 0.5, NP_DT[dt])
    tol = STEP_TOL[(dt, step_kernel)][0]
    err = max_rel_err(got, want)
    assert err <= tol, err
    np.testing.assert_array_equal(got[..., :n_in], s[..., :n_in])
    # cells that did not fire are copied bit for bit
    mask = oracle.fire_mask(42, 2, 0, shape, 0.5)
    np.testing.assert_array_equal(got[~mask], s[~mask])


@pytest.mark.parametrize("dt,ndim,n_in,shape", [("f32", 2, 3, (1, 40, 70)),
                                                ("f32", 3, 1, (6, 20, 18)),
                                                ("f16", 3, 3, (8, 12, 20)),
                                                ("f32", 3, 1, (40, 12, 40)),
                                                ("f32", 2, 3, (1, 140, 50)),
                                                ("f16", 3, 3, (40, 10, 36))])
def test_level_steps_match_oracle(gpu, step_kernel, dt, ndim, n_in, shape):
    rng = np.random.default_rng(12)
    w = rand_weights(rng, ndim)
    s = rng.normal(0, 1, shape + (C,)).astype(NP_DT[dt])
    steps = 9
    got, which = run_level_gpu(octnca.Model(ndim=ndim, n_in=n_in, dtype=dt, kernel=step_kernel),
                               s, w, 1, steps, 0.5, 3)
    assert which == steps % 2
    want = oracle.run_level(s, w, n_in, ndim, 1, steps, 3, 0.5, NP_DT[dt])
    tol = STEP_TOL[(dt, step_kernel)][1]
    assert max_rel_err(got, want) <= tol


@pytest.mark.parametrize("kernel", ["mfma", "mfma_rows", "mfma_tiles", "mfma_1step", "valu"])
@pytest.mark.parametrize("dt,ndim,n_in,c,h,shape", [
    ("f32", 2, 3, 12, 48, (1, 37, 45)), ("f32", 3, 1, 20, 100, (5, 9, 17)),
    ("f16", 2, 1, 20, 100, (1, 21, 30)), ("f16", 3, 3, 12, 48, (6, 11, 10)),
    ("f32", 3, 3, 12, 48, (4, 10, 12)), ("f16", 2, 3, 12, 48, (1, 16, 40)),
    ("f32", 2, 3, 20, 100, (1, 19, 70)), ("f32", 2, 1, 12, 48, (1, 33, 65)),
    ("f16", 3, 1, 20, 100, (7, 9, 33)), ("f32", 3, 3, 20, 100, (3, 5, 40)),
    ("f32", 2, 3, 12, 48, (1, 1, 1)), ("f16", 3, 3, 20, 100, (1, 1, 1)),
    ("f32", 3, 1, 12, 48, (9, 19, 70)), ("f32", 3, 3, 12, 48, (7, 17, 64))])
def test_other_model_sizes_match_oracle(gpu, kernel, dt, ndim, n_in, c, h, shape):
    """The ablation's model sizes C/H = 12/48 and 20/100 (supplement S10) on
    every kernel that serves them: 2D fp32 states of 12/48 on the row kernels
    ("mfma": one step per launch on levels this small, "mfma_rows": two steps
    per launch, "mfma_1step": one) or the generic tile kernel ("mfma_tiles"),
    3D fp32 states of 12/48 on the 3D step of 16/64 (rows on and off the
    8-cell grid), the other cases on the generic matrix-core kernel ("mfma"),
    and all on the vector kernel ("valu"): one step and nine steps against the
    oracle (several strips or tiles, ragged tails, a single cell), input
    channels unchanged, non-firing cells copied bit for bit."""
    if kernel in ("mfma_rows", "mfma_tiles", "mfma_1step") and (dt, ndim, c) != ("f32", 2, 12):
        pytest.skip("the same generic kernel as the 'mfma' case")
    rng = np.random.default_rng(13)
    w = rand_weights(rng, ndim, c=c, h=h)
    s = rng.normal(0, 1, shape + (c,)).astype(NP_DT[dt])
    model = octnca.Model(ndim=ndim, n_in=n_in, dtype=dt, channels=c, hidden=h, kernel=kernel)
    got, which = run_level_gpu(model, s, w, 2, 1, 0.5, 42)
    assert which == 1
    want = oracle.nca_step(s, w, n_in, ndim, 2, 0, 42, 0.5, NP_DT[dt])
    assert max_rel_err(got, want) <= STEP_TOL[(dt, kernel)][0]
    np.testing.assert_array_equal(got[..., :n_in], s[..., :n_in])
    mask = oracle.fire_mask(42, 2, 0, shape, 0.5)
    np.testing.assert_array_equal(got[~mask], s[~mask])
    got9, _ = run_level_gpu(model, s, w, 1, 9, 0.5, 3)
    want9 = oracle.run_level(s, w, n_in, ndim, 1, 9, 3, 0.5, NP_DT[dt])
    assert max_rel_err(got9, want9) <= STEP_TOL[(dt, kernel)][1]


def oracle_window_steps(s, w, n_in, ndim, level, steps, seed, rate, dt, box):
    """The oracle's ``steps`` steps of the cells in ``box`` ((z0, z1), (y0, y1),
    (x0, x1)) of the level held in ``s``, from a window that adds ``steps``
    halo cells on every side away from the level's border (light cone)."""
    grid = s.shape[:3]
    lo = [max(0, a - steps) for a, _ in box]
    hi = [min(n, b + steps) for (_, b), n in zip(box, grid)]
    win = s[lo[0]:hi[0], lo[1]:hi[1], lo[2]:hi[2]]
    for t in range(steps):
        win = oracle.nca_step(win, w, n_in, ndim, level, t, seed, rate, NP_DT[dt],
                              origin=tuple(lo), grid=grid)
    return win[tuple(slice(a - l, b - l) for (a, b), l in zip(box, lo))]


@pytest.mark.parametrize("dt,extent", [("f16", (300, 8, 24572)), ("f16", (300, 8, 24576)),
                                       ("f32", (300, 8, 24572)), ("f32", (300, 8, 24576))])
def test_long_3d_runs_match_oracle_on_windows(gpu, dt, extent):
    """Levels deep and wide enough that the 3D step streams runs of more than
    32 output planes (the launch's load model picks 151 planes for fp16 and 76
    for fp32 on these extents, with 768 columns), rows on and off the 8-cell
    grid (up to 38 fire evaluations per run): three steps against the
    oracle on windows at the grid's faces, at run boundaries of several run
    lengths and across a strip boundary."""
    rng = np.random.default_rng(31)
    w = rand_weights(rng, 3)
    n_in = 1
    d, h, wd = extent
    # a random block tiled over the level (cheap to build at 59 M cells)
    block = rng.normal(0, 1, (20, h, 256, C)).astype(NP_DT[dt])
    s = np.tile(block, (-(-d // 20), 1, -(-wd // 256), 1))[:d, :, :wd]
    s = np.ascontiguousarray(s)
    steps = 3
    got, which = run_level_gpu(octnca.Model(ndim=3, n_in=n_in, dtype=dt), s, w, 1, steps, 0.5, 9)
    assert which == steps % 2
    zs = [(0, 3), (74, 80), (97, 104), (150, 153), (197, 203), (295, 300)]
    xs = [(0, 36), (12270, 12322), (wd - 40, wd)]
    tol = STEP_TOL[(dt, "mfma")][1]
    for z in zs:
        for x in xs:
            box = (z, (0, h), x)
            want = oracle_window_steps(s, w, n_in, 3, 1, steps, 9, 0.5, dt, box)
            part = got[z[0]:z[1], :, x[0]:x[1]]
            assert max_rel_err(part, want) <= tol, (z, x)
            np.testing.assert_array_equal(part[..., :n_in], s[z[0]:z[1], :, x[0]:x[1], :n_in])


def test_zero_steps_leave_state(gpu):
    rng = np.random.default_rng(1)
    s = rng.normal(0, 1, (1, 9, 9, C)).astype(np.float32)
    got, which = run_level_gpu(octnca.Model(ndim=2, n_in=3), s, rand_weights(rng, 2), 0, 0, 0.5, 0)
    assert which == 0
    np.testing.assert_array_equal(got, s)


@pytest.mark.parametrize("ndim", [2, 3])
def test_fire_rate_zero_and_zero_w2_are_identity(gpu, step_kernel, ndim):
    rng = np.random.default_rng(2)
    shape = (1, 23, 41) if ndim == 2 else (5, 10, 12)
    s = rng.normal(0, 1, shape + (C,)).astype(np.float32)
    w = rand_weights(rng, ndim)
    m = octnca.Model(ndim=ndim, n_in=3, kernel=step_kernel)
    got, _ = run_level_gpu(m, s, w, 0, 3, 0.0, 5)
    np.testing.assert_array_equal(got, s)
    w.w2[:] = 0
    got, _ = run_level_gpu(m, s, w, 0, 3, 1.0, 5)
    np.testing.assert_array_equal(got, s)


@pytest.mark.parametrize("dt,ndim,n_in,shape", [("f32", 2, 3, (1, 30, 70)),
                                                ("f32", 3, 1, (6, 20, 40)),
                                                ("f16", 3, 3, (8, 12, 40)),
                                                ("f16", 2, 1, (1, 20, 50))])
def test_input_rows_of_w2_are_ignored(gpu, step_kernel, dt, ndim, n_in, shape):
    """The W2 rows of the input channels are part of the [C][H] array but
    their values never reach the state: the kernels read them and replace them
    by zero, so NaN there gives the same bits as zeros."""
    rng = np.random.default_rng(21)
    w = rand_weights(rng, ndim)
    s = rng.normal(0, 1, shape + (C,)).astype(NP_DT[dt])
    m = octnca.Model(ndim=ndim, n_in=n_in, dtype=dt, kernel=step_kernel)
    w.w2[:n_in] = 0
    ref, _ = run_level_gpu(m, s, w, 1, 3, 0.5, 8)
    w.w2[:n_in] = np.nan
    got, _ = run_level_gpu(m, s, w, 1, 3, 0.5, 8)
    np.testing.assert_array_equal(got, ref)
    assert np.isfinite(got).all()


@pytest.mark.parametrize("kernel", ["mfma", "valu"])
@pytest.mark.parametrize("dt,ndim,n_in,c,h", [("f32", 2, 3, 12, 48), ("f16", 3, 1, 20, 100)])
def test_input_rows_of_w2_are_ignored_other_sizes(gpu, kernel, dt, ndim, n_in, c, h):
    rng = np.random.default_rng(22)
    w = rand_weights(rng, ndim, c=c, h=h)
    shape = (1, 19, 40) if ndim == 2 else (5, 9, 36)
    s = rng.normal(0, 1, shape + (c,)).astype(NP_DT[dt])
    m = octnca.Model(ndim=ndim, n_in=n_in, dtype=dt, channels=c, hidden=h, kernel=kernel)
    w.w2[:n_in] = 0
    ref, _ = run_level_gpu(m, s, w, 1, 3, 0.5, 8)
    w.w2[:n_in] = np.nan
    got, _ = run_level_gpu(m, s, w, 1, 3, 0.5, 8)
    np.testing.assert_array_equal(got, ref)
    assert np.isfinite(got).all()


def test_translation_equivariance_on_gpu(gpu, step_kernel):
    """With every cell firing, shifting the input shifts the output (cells far
    enough from the border)."""
    rng = np.random.default_rng(4)
    w = rand_weights(rng, 2)
    m = octnca.Model(ndim=2, n_in=3, kernel=step_kernel)
    base = rng.normal(0, 1, (1, 48, 64, C)).astype(np.float32)
    shifted = np.roll(base, (5, 9), axis=(1, 2))
    a, _ = run_level_gpu(m, base, w, 0, 4, 1.0, 0)
    b, _ = run_level_gpu(m, shifted, w, 0, 4, 1.0, 0)
    r = 4
    np.testing.assert_allclose(b[:, 5 + r:48 - r, 9 + r:64 - r],
                               a[:, r:48 - 5 - r, r:64 - 9 - r], rtol=0, atol=0)


def test_step_is_deterministic(gpu, step_kernel):
    rng = np.random.default_rng(6)
    w = rand_weights(rng, 3)
    s = rng.normal(0, 1, (9, 17, 19, C)).astype(np.float32)
    m = octnca.Model(ndim=3, n_in=1, kernel=step_kernel)
    a, _ = run_level_gpu(m, s, w, 0, 5, 0.5, 1)
    b, _ = run_level_gpu(m, s, w, 0, 5, 0.5, 1)
    np.testing.assert_array_equal(a, b)


def test_split_bf16_kernel_on_fp16_states(gpu):
    rng = np.random.default_rng(13)
    w = rand_weights(rng, 3)
    s = rng.normal(0, 1, (6, 11, 35, C)).astype(np.float16)
    got, _ = run_level_gpu(octnca.Model(ndim=3, n_in=3, dtype="f16", kernel="mfma_bf16x3"), s, w,
                           0, 4, 0.5, 8)
    want = oracle.run_level(s, w, 3, 3, 0, 4, 8, 0.5, np.float16)
    assert max_rel_err(got, want) <= 5e-3


def test_scaled_fp16_mlp_keeps_large_fp32_states_in_range(gpu):
    """The default MLP of fp32 states rounds its activations to fp16 after a
    2^-8 scaling: states and hidden units far beyond fp16's 65504 stay finite
    and as accurate as at unit scale (without the scaling the hidden units
    here, ~1e5-1e6, would overflow fp16)."""
    rng = np.random.default_rng(17)
    w = rand_weights(rng, 2)
    s = rng.normal(0, 1, (1, 24, 40, C)).astype(np.float32)
    m = octnca.Model(ndim=2, n_in=3)
    for scale in (1.0, 2.0 ** 17):
        got, _ = run_level_gpu(m, s * np.float32(scale), w, 1, 1, 0.5, 3)
        want = oracle.run_level(s * np.float32(scale), w, 3, 2, 1, 1, 3, 0.5, np.float32)
        assert np.all(np.isfinite(got))
        assert max_rel_err(got, want) <= STEP_TOL[("f32", "mfma")][0]


def test_fp16_operands_refused_for_fp32_states(gpu):
    """fp16 MLP operands are not offered for fp32 states: the call is
    refused before anything is enqueued."""
    s = np.zeros((1, 8, 8, C), np.float32)
    b0 = dev(s)
    b1 = torch.empty_like(b0)
    w = upload_weights([rand_weights(np.random.default_rng(0), 2)])[0]
    with pytest.raises(octnca.OctreeNCAError):
        octnca.octree_nca_run_level(octnca.Model(ndim=2, n_in=3, kernel="mfma_f16"), b0, b1, w,
                                    0, 1, 0.5, 0)
