"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects invalid arguments before it enqueues anything
(every call below fails validation, so no HIP call is made)."""
import ctypes
import math
import os
import re

import pytest

import paper_2508_06993_amd as octnca
from paper_2508_06993_amd import _Extent, _LevelWeights, _Model

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "octree_nca.h")

EINVAL, EUNSUP, ESHAPE, ESPACE = (octnca.OCTNCA_EINVAL, octnca.OCTNCA_EUNSUPPORTED,
                                  octnca.OCTNCA_ESHAPE, octnca.OCTNCA_ESPACE)
FAKE = ctypes.c_void_p(0x7f0000001000)    # never dereferenced: validation fails first
FAKE2 = ctypes.c_void_p(0x7f0000900000)


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(
        r"^(?:int|int32_t|size_t|const char \*)\s*(octree_nca_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib(library_path):
    return octnca.lib()


def model(ndim=2, c=16, h=64, n_in=3, dt=0):
    return ctypes.byref(_Model(ndim, c, h, n_in, dt))


def weights():
    return ctypes.byref(_LevelWeights(FAKE, FAKE, FAKE, FAKE, FAKE))


def test_header_declares_the_four_named_entry_points():
    names = declared_functions()
    for n in ("octree_nca_build_pyramid", "octree_nca_run_level", "octree_nca_upsample",
              "octree_nca_infer"):
        assert n in names
    assert set(names) == set(octnca.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(lib, library_path):
    raw = ctypes.CDLL(library_path)
    for name in declared_functions():
        assert hasattr(raw, name), name


def test_version_and_strerror(lib):
    declared = int(re.search(r"#define OCTNCA_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert lib.octree_nca_abi_version() == declared == 5
    for st in (0, -1, -2, -3, -4, -5):
        assert lib.octree_nca_strerror(st).decode() not in ("", "unknown status")
    assert lib.octree_nca_strerror(17).decode() == "unknown status"


@pytest.mark.parametrize("m", [dict(c=12), dict(h=48), dict(n_in=2), dict(ndim=4),
                               dict(dt=7), dict(ndim=1)])
def test_unsupported_models(lib, m):
    st = lib.octree_nca_run_level(model(**m), FAKE, FAKE2, _Extent(1, 8, 8), weights(), 0, 1,
                                  0.5, 0, None, None)
    assert st == EUNSUP


def test_null_model(lib):
    assert lib.octree_nca_run_level(None, FAKE, FAKE2, _Extent(1, 8, 8), weights(), 0, 1, 0.5,
                                    0, None, None) == EINVAL


@pytest.mark.parametrize("ext,nd", [((1, 0, 8), 2), ((1, 8, -1), 2), ((2, 8, 8), 2),
                                    ((0, 4, 4), 3), ((1, 1 << 31, 4), 2)])
def test_bad_extents(lib, ext, nd):
    st = lib.octree_nca_run_level(model(ndim=nd), FAKE, FAKE2, _Extent(*ext), weights(), 0, 1,
                                  0.5, 0, None, None)
    assert st == ESHAPE


@pytest.mark.parametrize("rate", [-0.1, 1.0001, math.nan, math.inf])
def test_fire_rate_outside_unit_interval(lib, rate):
    assert lib.octree_nca_run_level(model(), FAKE, FAKE2, _Extent(1, 8, 8), weights(), 0, 1,
                                    rate, 0, None, None) == EINVAL
    m = (ctypes.c_uint8 * 1)()
    assert lib.octree_nca_fire_mask(0, 0, 0, _Extent(1, 4, 4), rate, FAKE, None) == EINVAL


def test_run_level_argument_checks(lib):
    e = _Extent(1, 8, 8)
    assert lib.octree_nca_run_level(model(), None, FAKE2, e, weights(), 0, 1, 0.5, 0, None,
                                    None) == EINVAL
    assert lib.octree_nca_run_level(model(), FAKE, FAKE, e, weights(), 0, 1, 0.5, 0, None,
                                    None) == EINVAL   # in place is not allowed
    overlapping = ctypes.c_void_p(FAKE.value + 64)
    assert lib.octree_nca_run_level(model(), FAKE, overlapping, e, weights(), 0, 1, 0.5, 0,
                                    None, None) == EINVAL
    assert lib.octree_nca_run_level(model(), FAKE, FAKE2, e, weights(), 0, -1, 0.5, 0, None,
                                    None) == EINVAL
    assert lib.octree_nca_run_level(model(), FAKE, FAKE2, e, weights(), -1, 1, 0.5, 0, None,
                                    None) == EINVAL
    bad = ctypes.byref(_LevelWeights(FAKE, FAKE, None, FAKE, FAKE))
    assert lib.octree_nca_run_level(model(), FAKE, FAKE2, e, bad, 0, 1, 0.5, 0, None,
                                    None) == EINVAL


def test_cell_count_limit_has_no_overflow(lib):
    """2^36 cells per level at most: an extent whose cell count exceeds it is
    rejected also where d * h * w does not fit 64 bits (64 x 2^30 x (2^28 + 1)
    is 2^64 + 2^36 cells, which a 64-bit product wraps to exactly 2^36)."""
    m3 = model(ndim=3, n_in=1)
    assert lib.octree_nca_workspace_bytes(m3, _Extent(64, 1 << 30, (1 << 28) + 1), 1, None, 1) == 0
    assert lib.octree_nca_workspace_bytes(m3, _Extent(64, 1 << 30, 1 << 30), 1, None, 1) == 0
    assert lib.octree_nca_workspace_bytes(m3, _Extent(64, 1 << 30, 2), 1, None, 1) == 0
    assert lib.octree_nca_workspace_bytes(m3, _Extent(64, 1 << 20, 1 << 11), 1, None, 1) == 0
    assert lib.octree_nca_workspace_bytes(m3, _Extent(64, 1 << 20, 1 << 10), 1, None, 1) > 0
    assert lib.octree_nca_workspace_bytes(m3, _Extent(64, 1 << 20, 1 << 9), 1, None, 1) > 0


def test_batch_size_limit(lib):
    """A batch whose states would exceed 2^48 bytes is rejected before any
    pointer arithmetic (2^31 - 1 images of 2^20 x 2^10 cells)."""
    assert lib.octree_nca_infer_batch(model(), FAKE, (1 << 31) - 1, _Extent(1, 1 << 20, 1 << 10),
                                      1, None, weights(), (ctypes.c_int32 * 1)(1), 0.5, 0, FAKE2,
                                      1 << 40, None, None, None) == EINVAL


def test_pyramid_and_upsample_shape_checks(lib):
    f = (ctypes.c_int32 * 6)(1, 2, 2, 1, 2, 2)
    imgs = (ctypes.c_void_p * 2)(FAKE, FAKE2)
    # 10 is not divisible by 4
    assert lib.octree_nca_build_pyramid(model(), FAKE, _Extent(1, 8, 10), 3, f, imgs,
                                        None) == ESHAPE
    f2d_bad = (ctypes.c_int32 * 3)(2, 2, 2)      # 2D model cannot pool depth
    assert lib.octree_nca_build_pyramid(model(), FAKE, _Extent(1, 8, 8), 2, f2d_bad, imgs,
                                        None) == ESHAPE
    f0 = (ctypes.c_int32 * 3)(1, 0, 2)
    assert lib.octree_nca_upsample(model(), FAKE, _Extent(1, 4, 4), f0, FAKE2, FAKE,
                                   None) == ESHAPE
    f1 = (ctypes.c_int32 * 3)(1, 2, 2)
    # fine state overlapping the coarse state
    assert lib.octree_nca_upsample(model(), FAKE, _Extent(1, 4, 4), f1, FAKE2,
                                   ctypes.c_void_p(FAKE.value + 16), None) == EINVAL
    assert lib.octree_nca_build_pyramid(model(), FAKE, _Extent(1, 8, 8), 0, f, imgs,
                                        None) == EINVAL


def test_workspace_bytes_layout(lib):
    f = (ctypes.c_int32 * 6)(1, 2, 2, 1, 2, 2)
    ext = _Extent(1, 64, 64)
    al = lambda n: (n + 255) // 256 * 256
    img = al(32 * 32 * 3 * 4) + al(16 * 16 * 3 * 4)
    state = al(64 * 64 * 16 * 4)
    assert lib.octree_nca_workspace_bytes(model(), ext, 3, f, 1) == img + state
    assert lib.octree_nca_workspace_bytes(model(), ext, 3, f, 0) == img + 2 * state
    assert lib.octree_nca_workspace_bytes(model(dt=1), ext, 3, f, 1) == \
        al(32 * 32 * 3 * 2) + al(16 * 16 * 3 * 2) + al(64 * 64 * 16 * 2)
    assert lib.octree_nca_workspace_bytes(model(), _Extent(1, 63, 64), 3, f, 1) == 0


def test_other_model_sizes_are_accepted(lib):
    """C/H = 12/48 and 20/100 (the paper's ablation sizes) are supported: the
    state buffers of the workspace scale with C; other pairs are refused."""
    f = (ctypes.c_int32 * 3)(1, 2, 2)
    ext = _Extent(1, 64, 64)
    al = lambda n: (n + 255) // 256 * 256
    img = al(32 * 32 * 3 * 4)
    for c, h in ((12, 48), (16, 64), (20, 100)):
        assert lib.octree_nca_workspace_bytes(model(c=c, h=h), ext, 2, f, 0) == \
            img + 2 * al(64 * 64 * c * 4)
    for c, h in ((12, 64), (20, 64), (16, 48), (8, 32)):
        assert lib.octree_nca_workspace_bytes(model(c=c, h=h), ext, 2, f, 0) == 0
    # the K-class readout range follows C
    assert lib.octree_nca_readout_classes(model(c=12, h=48), FAKE, _Extent(1, 8, 8), 10, FAKE2,
                                          None) == EINVAL


def test_infer_rejects_small_workspace_and_bad_steps(lib):
    L = 3
    f = (ctypes.c_int32 * 6)(1, 2, 2, 1, 2, 2)
    ws = (_LevelWeights * L)(*[_LevelWeights(FAKE, FAKE, FAKE, FAKE, FAKE)] * L)
    steps = (ctypes.c_int32 * L)(10, 10, 10)
    ext = _Extent(1, 64, 64)
    need = lib.octree_nca_workspace_bytes(model(), ext, L, f, 1)
    final = ctypes.c_void_p(0x7f1000000000)
    image = ctypes.c_void_p(0x7f2000000000)
    wsp = ctypes.c_void_p(0x7f3000000000)
    assert lib.octree_nca_infer(model(), image, ext, L, f, ws, steps, 0.5, 0, wsp, need - 1,
                                final, None, None, None) == ESPACE
    bad_steps = (ctypes.c_int32 * L)(10, -1, 10)
    assert lib.octree_nca_infer(model(), image, ext, L, f, ws, bad_steps, 0.5, 0, wsp, need,
                                final, None, None, None) == EINVAL
    # final state inside the workspace
    assert lib.octree_nca_infer(model(), image, ext, L, f, ws, steps, 0.5, 0, wsp, need,
                                ctypes.c_void_p(wsp.value + 256), None, None, None) == EINVAL


@pytest.mark.parametrize("classes,n_in,expect", [(1, 3, EINVAL), (0, 3, EINVAL),
                                                  (14, 3, EINVAL), (16, 1, EINVAL),
                                                  (-2, 3, EINVAL)])
def test_readout_classes_range(lib, classes, n_in, expect):
    st = lib.octree_nca_readout_classes(model(n_in=n_in), FAKE, _Extent(1, 8, 8), classes, FAKE2,
                                        None)
    assert st == expect


def test_readout_classes_other_checks(lib):
    assert lib.octree_nca_readout_classes(model(), None, _Extent(1, 8, 8), 2, FAKE2,
                                          None) == EINVAL
    assert lib.octree_nca_readout_classes(model(), FAKE, _Extent(1, 8, 8), 2, None,
                                          None) == EINVAL
    assert lib.octree_nca_readout_classes(model(), FAKE, _Extent(2, 8, 8), 2, FAKE2,
                                          None) == ESHAPE
    assert lib.octree_nca_readout_classes(model(c=12), FAKE, _Extent(1, 8, 8), 2, FAKE2,
                                          None) == EUNSUP


def test_infer_batch_argument_checks(lib):
    L = 3
    f = (ctypes.c_int32 * 6)(1, 2, 2, 1, 2, 2)
    ws = (_LevelWeights * L)(*[_LevelWeights(FAKE, FAKE, FAKE, FAKE, FAKE)] * L)
    steps = (ctypes.c_int32 * L)(10, 10, 10)
    ext = _Extent(1, 64, 64)
    need = lib.octree_nca_workspace_bytes(model(), ext, L, f, 1)
    images = ctypes.c_void_p(0x7f2000000000)
    finals = ctypes.c_void_p(0x7f1000000000)
    wsp = ctypes.c_void_p(0x7f3000000000)
    image_bytes, state_bytes = 64 * 64 * 3 * 4, 64 * 64 * 16 * 4

    def call(batch=2, finals=finals, segs=None, wsp=wsp, n=need, steps=steps, images=images):
        return lib.octree_nca_infer_batch(model(), images, batch, ext, L, f, ws, steps, 0.5, 0,
                                          wsp, n, finals, segs, None)
    assert call(batch=0) == EINVAL
    assert call(batch=-3) == EINVAL
    assert call(images=None) == EINVAL
    assert call(n=need - 1) == ESPACE
    assert call(steps=(ctypes.c_int32 * L)(10, -1, 10)) == EINVAL
    # the second image's final state overlaps the first image
    assert call(finals=ctypes.c_void_p(images.value + image_bytes - state_bytes)) == EINVAL
    # segmentation of image 1 inside the workspace
    assert call(segs=ctypes.c_void_p(wsp.value + 64)) == EINVAL
    # images inside the workspace
    assert call(images=ctypes.c_void_p(wsp.value + 512)) == EINVAL
    # an unsupported model is reported before anything else
    assert lib.octree_nca_infer_batch(model(c=12), images, 2, ext, L, f, ws, steps, 0.5, 0, wsp,
                                      need, finals, None, None) == EUNSUP


def test_first_level_steps_matches_oracle(lib):
    import oracle
    for alpha in (0.0, 0.5, 1.0, 1.5, 2.0, 0.3, 3.7):
        for ext in ((1, 352, 512), (24, 80, 80), (450, 15, 27), (1, 1, 1), (7, 3, 5)):
            assert lib.octree_nca_first_level_steps(alpha, _Extent(*ext)) == \
                oracle.first_level_steps(alpha, ext), (alpha, ext)
    assert octnca.octree_nca_first_level_steps(1.0, (1, 352, 512)) == 512
    for alpha, ext in ((-1.0, (1, 4, 4)), (math.nan, (1, 4, 4)), (math.inf, (1, 4, 4)),
                       (1.0, (1, 0, 4)), (1.0, (-1, 4, 4)), (3e9, (1, 4, 4))):
        assert lib.octree_nca_first_level_steps(alpha, _Extent(*ext)) == -1


def test_python_binding_refuses_host_tensors(lib):
    import torch
    m = octnca.Model(ndim=2, n_in=3)
    with pytest.raises(octnca.OctreeNCAError):
        octnca.octree_nca_readout(m, torch.zeros(1, 4, 4, 16), torch.zeros(1, 4, 4,
                                                                            dtype=torch.uint8))


# ---------------------------------------------------------------------------
# training entry points (fp32 states only): validation before any launch
# ---------------------------------------------------------------------------

from paper_2508_06993_amd import _LevelGrads   # noqa: E402


def grads():
    return ctypes.byref(_LevelGrads(FAKE, FAKE, FAKE, FAKE, FAKE))


def bwd_ws_floats(ext, c=16, h=64, ndim=2):
    """G' + gS and gP (C floats per cell each), and one row of weight-gradient
    sums per block of the per-cell backward (2 x 32 cells in 2D, 2 x 4 x 8 in
    3D)."""
    d, hh, w = ext
    cells = d * hh * w
    taps = 27 if ndim == 3 else 9
    tz, ty, tx = (2, 4, 8) if ndim == 3 else (1, 2, 32)
    blocks = -(-d // tz) * -(-hh // ty) * -(-w // tx)
    return 2 * cells * c + blocks * (3 * c * h + h + c + c * taps)


def test_step_backward_workspace_bytes(lib):
    assert lib.octree_nca_step_backward_workspace_bytes(model(), _Extent(1, 8, 10)) == \
        4 * bwd_ws_floats((1, 8, 10))
    assert lib.octree_nca_step_backward_workspace_bytes(model(ndim=3, n_in=1), _Extent(3, 5, 7)) \
        == 4 * bwd_ws_floats((3, 5, 7), ndim=3)
    assert lib.octree_nca_step_backward_workspace_bytes(model(ndim=4), _Extent(1, 8, 8)) == 0


def step_bwd(lib, m=None, state=FAKE, gout=FAKE2, ext=(1, 8, 8), level=0, step=0, rate=0.5,
             gin=ctypes.c_void_p(0x7f0010000000), gr=None, ws=ctypes.c_void_p(0x7f0020000000),
             ws_bytes=1 << 30):
    return lib.octree_nca_step_backward(m if m is not None else model(), state, gout,
                                        _Extent(*ext), weights(), level, step, rate, 0, gin,
                                        gr if gr is not None else grads(), ws, ws_bytes, None)


def test_step_backward_rejects_bad_arguments(lib):
    assert step_bwd(lib, m=model(dt=1)) == EUNSUP                 # fp16 states
    assert step_bwd(lib, state=None) == EINVAL
    assert step_bwd(lib, gr=ctypes.byref(_LevelGrads(FAKE, None, FAKE, FAKE, FAKE))) == EINVAL
    assert step_bwd(lib, step=-1) == EINVAL
    assert step_bwd(lib, rate=1.5) == EINVAL
    assert step_bwd(lib, ws_bytes=100) == ESPACE
    assert step_bwd(lib, gin=FAKE) == EINVAL                      # grad_in overlaps state
    assert step_bwd(lib, ws=FAKE2) == EINVAL                      # workspace overlaps grad_out
    assert step_bwd(lib, ext=(1, 0, 8)) == ESHAPE


def test_upsample_backward_rejects_bad_arguments(lib):
    f = (ctypes.c_int32 * 3)(1, 2, 2)
    assert lib.octree_nca_upsample_backward(model(dt=1), FAKE, _Extent(1, 4, 4), f, FAKE2,
                                            None) == EUNSUP
    assert lib.octree_nca_upsample_backward(model(), None, _Extent(1, 4, 4), f, FAKE2,
                                            None) == EINVAL
    bad = (ctypes.c_int32 * 3)(2, 2, 2)                          # fz != 1 in 2D
    assert lib.octree_nca_upsample_backward(model(), FAKE, _Extent(1, 4, 4), bad, FAKE2,
                                            None) == ESHAPE
    assert lib.octree_nca_upsample_backward(model(), FAKE, _Extent(1, 4, 4), f, FAKE,
                                            None) == EINVAL     # in place


def test_readout_mse_rejects_bad_arguments(lib):
    assert lib.octree_nca_readout_mse_workspace_bytes(_Extent(1, 16, 20)) == 8 * 2
    assert lib.octree_nca_readout_mse_workspace_bytes(_Extent(1, 0, 20)) == 0
    ws = ctypes.c_void_p(0x7f0030000000)
    assert lib.octree_nca_readout_mse(model(), FAKE, FAKE2, _Extent(1, 16, 20),
                                      ctypes.c_void_p(0x7f0010000000), ws, ws, 8,
                                      None) == ESPACE
    assert lib.octree_nca_readout_mse(model(dt=1), FAKE, FAKE2, _Extent(1, 16, 20),
                                      ctypes.c_void_p(0x7f0010000000), ws, ws, 64,
                                      None) == EUNSUP
    assert lib.octree_nca_readout_mse(model(), FAKE, FAKE2, _Extent(1, 16, 20), None, ws, ws,
                                      64, None) == EINVAL


def test_train_workspace_and_step_validation(lib):
    f = (ctypes.c_int32 * 3)(1, 2, 2)
    steps = (ctypes.c_int32 * 2)(3, 2)
    n = lib.octree_nca_train_workspace_bytes(model(), _Extent(1, 8, 8), 2, f, steps)
    assert n > 4 * (4 * 64 * 16 + 3 * 16 * 16)        # at least the tape of both levels
    assert lib.octree_nca_train_workspace_bytes(model(dt=1), _Extent(1, 8, 8), 2, f, steps) == 0
    neg = (ctypes.c_int32 * 2)(3, -1)
    assert lib.octree_nca_train_workspace_bytes(model(), _Extent(1, 8, 8), 2, f, neg) == 0
    ws = (_LevelWeights * 2)(*[_LevelWeights(FAKE, FAKE, FAKE, FAKE, FAKE)] * 2)
    gs = (_LevelGrads * 2)(*[_LevelGrads(FAKE, FAKE, FAKE, FAKE, FAKE)] * 2)
    big = ctypes.c_void_p(0x7f4000000000)
    args = lambda wsb: (model(), FAKE, _Extent(1, 8, 8), 2, f, ws, steps, 0.5, 0, FAKE2, big,
                        wsb, gs, ctypes.c_void_p(0x7f0050000000), None, None)
    assert lib.octree_nca_train_step(*args(n - 1)) == ESPACE
    assert lib.octree_nca_train_step(model(), FAKE, _Extent(1, 8, 8), 2, f, ws, steps, 0.5, 0,
                                     FAKE2, big, n, gs, None, None, None) == EINVAL


def test_infer_launches_counts_two_step_launches():
    """Host query of the launches octree_nca_infer enqueues: on the 184.5 MP
    pyramid the three large levels run their 20 steps in 10 two-step launches,
    the first fused with the upsample; an odd count adds one single step; the
    smaller levels and the one-step selection run one launch per step."""
    m = octnca.Model(ndim=2, n_in=3)
    f = [(1, 2, 2)] * 5
    assert octnca.octree_nca_infer_launches(m, (1, 11264, 16384), f, [20] * 6) == \
        [10, 10, 10, 20, 20, 20]
    assert octnca.octree_nca_infer_launches(m, (1, 11264, 16384), f, [19, 1, 2, 20, 20, 20]) == \
        [10, 1, 1, 20, 20, 20]
    one = octnca.Model(ndim=2, n_in=3, kernel="mfma_1step")
    assert octnca.octree_nca_infer_launches(one, (1, 11264, 16384), f, [20] * 6) == [20] * 6
    rows = octnca.Model(ndim=2, n_in=3, kernel="mfma_rows")
    assert octnca.octree_nca_infer_launches(rows, (1, 64, 64), [(1, 2, 2)] * 2, [5, 4, 0]) == \
        [3, 2, 0]
    valu = octnca.Model(ndim=2, n_in=3, kernel="valu")
    assert octnca.octree_nca_infer_launches(valu, (1, 64, 64), [(1, 2, 2)] * 2, [5, 4, 3]) == \
        [5, 4, 3]
    # the plan is a function of the arguments: the level of 2048 two-step work
    # items (1920 = 64 strips of 30 cells, 4096 rows = 32 runs of 128) pairs,
    # one of 1984 items does not, on any device
    assert octnca.octree_nca_infer_launches(m, (1, 4096, 1920), [], [20]) == [10]
    assert octnca.octree_nca_infer_launches(m, (1, 3968, 1920), [], [20]) == [20]
    with pytest.raises(octnca.OctreeNCAError):
        octnca.octree_nca_infer_launches(m, (1, 64, 64), [(1, 2, 2)] * 2, [5, -1, 3])


def test_infer_launches_of_the_other_model_sizes():
    """The 12/48 model's fp32 2D steps take the row kernels of 16/64, two steps
    per launch included; its fp16 steps, its 3D steps and the 20/100 model run
    one step per launch (no upsample fusion in 3D fp32 and on the generic
    kernel, so each level but the coarsest adds none)."""
    f = [(1, 2, 2)] * 5
    c12 = octnca.Model(ndim=2, n_in=3, channels=12, hidden=48)
    assert octnca.octree_nca_infer_launches(c12, (1, 11264, 16384), f, [20] * 6) == \
        [10, 10, 10, 20, 20, 20]
    c12_1 = octnca.Model(ndim=2, n_in=3, channels=12, hidden=48, kernel="mfma_1step")
    assert octnca.octree_nca_infer_launches(c12_1, (1, 11264, 16384), f, [20] * 6) == [20] * 6
    c12_h = octnca.Model(ndim=2, n_in=3, dtype="f16", channels=12, hidden=48)
    assert octnca.octree_nca_infer_launches(c12_h, (1, 4096, 1920), [], [20]) == [20]
    c20 = octnca.Model(ndim=2, n_in=3, channels=20, hidden=100)
    assert octnca.octree_nca_infer_launches(c20, (1, 11264, 16384), f, [20] * 6) == [20] * 6
    c12_3 = octnca.Model(ndim=3, n_in=1, channels=12, hidden=48)
    assert octnca.octree_nca_infer_launches(c12_3, (24, 320, 320), [(1, 2, 2)] * 2,
                                            [20] * 3) == [20] * 3


def test_model_kernel_fields_are_checked(lib):
    """The step-kernel fields of octnca_model: values outside their enums are
    EINVAL, combinations no kernel implements EUNSUPPORTED; checked before
    anything else, with no launch."""
    def m(mlp=0, layout=0, spl=0, c=16, h=64, dt=0):
        return ctypes.byref(_Model(2, c, h, 3, dt, mlp, layout, spl))
    steps = (ctypes.c_int32 * 1)(3)
    out = (ctypes.c_int32 * 1)()
    f = (ctypes.c_int32 * 3)(1, 1, 1)
    call = lambda mm: lib.octree_nca_infer_launches(mm, _Extent(1, 8, 8), 1, f, steps, out)
    assert call(m()) == 0 and out[0] == 3                      # host-only query
    for bad in (m(mlp=6), m(mlp=-1), m(layout=3), m(spl=2), m(spl=-1)):
        assert call(bad) == EINVAL
    assert call(m(mlp=octnca.OCTNCA_MLP_F16)) == EUNSUP             # fp16 operands, fp32 states
    assert call(m(mlp=octnca.OCTNCA_MLP_F16S, dt=1)) == EUNSUP      # split operands, fp16 states
    assert call(m(mlp=octnca.OCTNCA_MLP_F32, c=12, h=48)) == EUNSUP # MFMA only for 16 / 64
    assert call(m(mlp=octnca.OCTNCA_MLP_VALU, c=12, h=48)) == 0     # vector kernel: accepted
    for name in octnca.KERNEL_NAMES:
        octnca.kernel_fields(name)
    assert octnca.kernel_fields("mfma_rows,mfma_1step") == {
        "mlp": 0, "layout2d": octnca.OCTNCA_LAYOUT_ROWS, "steps_per_launch": 1}
    with pytest.raises(ValueError):
        octnca.kernel_fields("mfma_fast")


def test_run_level_result_parity_is_steps_mod_2(lib):
    """run_level reports where its result is without a device: validation of
    every argument happens first, so an invalid call leaves the flag alone; the
    documented rule is steps % 2 for every kernel (checked on the GPU)."""
    res = ctypes.c_int32(7)
    ext = _Extent(1, 8, 8)
    assert lib.octree_nca_run_level(model(), FAKE, FAKE2, ext, weights(), 0, -1, 0.5, 0,
                                    ctypes.byref(res), None) == EINVAL
    assert res.value == 7


def test_build_stamp_tracks_sources(library_path, monkeypatch):
    """The library carries a stamp of the sources, headers and flags it was
    built from; the test session rebuilds whenever the stamp differs."""
    from paper_2508_06993_amd import build as b
    assert b.is_current()
    assert b.source_stamp() == b.source_stamp()
    monkeypatch.setattr(b, "COMMON_FLAGS", b.COMMON_FLAGS + ["-DSTAMP_PROBE"])
    assert not b.is_current()


def test_infer_static_validates_before_anything(lib):
    """octree_nca_infer_static checks its arguments (final_state required) and
    the workspace need against the static array before it looks the array
    up or enqueues anything."""
    f = (ctypes.c_int32 * 3)(1, 2, 2)
    steps = (ctypes.c_int32 * 2)(2, 2)
    ws = (_LevelWeights * 2)(*[_LevelWeights(FAKE, FAKE, FAKE, FAKE, FAKE)] * 2)
    call = lambda m, ext, final: lib.octree_nca_infer_static(m, FAKE, _Extent(*ext), 2, f, ws,
                                                            steps, 0.5, 0, final, None, None)
    assert call(model(), (1, 64, 64), None) == EINVAL
    assert call(model(), (1, 1024, 1024), FAKE2) == ESPACE       # 64 MiB state + pyramid
    assert call(model(c=13), (1, 64, 64), FAKE2) == EUNSUP
    assert call(model(), (1, 63, 64), FAKE2) == ESHAPE
    need = lib.octree_nca_workspace_bytes(model(), _Extent(1, 1024, 1024), 2, f, 1)
    assert need > octnca.OCTNCA_STATIC_SCRATCH_BYTES
    hdr = open(HEADER).read()
    assert re.search(r"#define OCTNCA_STATIC_SCRATCH_BYTES \(\(size_t\)64 << 20\)", hdr)
    assert octnca.OCTNCA_STATIC_SCRATCH_BYTES == 64 << 20
