"""Plain CPU oracle for OctreeNCA inference (arXiv 2508.06993).

TEST INFRASTRUCTURE.  This module is the slow, obviously correct reference
that the GPU path is checked against.  Only tests, the smoke check and the
benchmark's CPU-baseline leg may import it; the product path never does.  It
shares no code with the HIP library.

Arithmetic is float64 throughout.  Every stored quantity (pyramid images, the
state after each step, after initialisation and after each upsampling) is
rounded to the storage type of the workload (float32, or float16 with
round-to-nearest-even), because the paper keeps the state in device tensors
between steps (supplement S6, Listings 2 and 3).

Layout: every image/state is an array [D][H][W][channels]; a 2D workload has
D = 1 and uses 3x3 taps, a 3D (or 2D+t) workload uses 3x3x3 taps.  Level 0 is
the finest level, level L-1 the coarsest.

What is computed, and where the paper states it:

* pyramid: each coarser level is the mean of the finer level over one octree
  node (Sec. 3.2, "Repeated hidden channel upscaling"; supplement S7 table of
  level resolutions for the pooling factors);
* coarsest state: image in the first n_in channels, zeros elsewhere (Sec. 3.1,
  first n channels hold the input, the rest are hidden);
* between levels: nearest-neighbour upsampling of the state, then the level's
  image re-injected into the input channels (Sec. 3.2; supplement S6,
  Listings 2 and 3);
* one NCA step (Sec. 3.1; supplement S3, Listing 1): depthwise convolution of
  each channel with its learned 3x3(x3) kernel plus bias, concatenated after
  the cell's own state, a linear layer to the hidden size with bias, ReLU, a
  linear layer to the hidden channels without bias, multiplied by the cell's
  stochastic fire bit and added to the state; computed out of place
  (supplement S3);
* readout: two-class argmax over the last two channels (segmentation is
  predicted in the last hidden channel of the finest level, Sec. 3.2).

Readings taken where the paper is silent or ambiguous (each is listed with its
reason in the design notes): average pooling for the image pyramid, zero
padding, cross-correlation tap order, feature order [state, perception],
biases placed as the printed parameter counts require, one fire bit per cell
drawn from Philox4x64-10 (one 32-bit half of an output word per cell), argmax
ties resolved to the lower channel.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

from .philox import philox4x64

Box = Tuple[Tuple[int, int], Tuple[int, int], Tuple[int, int]]  # ((z0,z1),(y0,y1),(x0,x1))


# --------------------------------------------------------------------------
# storage
# --------------------------------------------------------------------------

def to_storage(x: np.ndarray, dtype) -> np.ndarray:
    """Round float64 values to the storage type (round to nearest even)."""
    return np.asarray(x, dtype=np.float64).astype(dtype)


# --------------------------------------------------------------------------
# pyramid (Sec. 3.2; supplement S7 table of octree level resolutions)
# --------------------------------------------------------------------------

def pool(image: np.ndarray, factor: Sequence[int], dtype) -> np.ndarray:
    """Next coarser level: I_{l+1}[z,y,x,c] = mean of I_l over the block
    [fz*z, fz*z+fz) x [fy*y, fy*y+fy) x [fx*x, fx*x+fx)."""
    fz, fy, fx = factor
    d, h, w, c = image.shape
    if d % fz or h % fy or w % fx:
        raise ValueError(f"extent {(d, h, w)} not divisible by factor {tuple(factor)}")
    blocks = image.astype(np.float64).reshape(d // fz, fz, h // fy, fy, w // fx, fx, c)
    mean = blocks.sum(axis=(1, 3, 5)) / float(fz * fy * fx)
    return to_storage(mean, dtype)


def build_pyramid(image: np.ndarray, factors: Sequence[Sequence[int]], dtype) -> List[np.ndarray]:
    """[I_0 (finest, the input itself), I_1, ..., I_{L-1}]."""
    levels = [np.asarray(image, dtype=dtype)]
    for f in factors:
        levels.append(pool(levels[-1], f, dtype))
    return levels


# --------------------------------------------------------------------------
# level transitions (Sec. 3.1, Sec. 3.2; supplement S6, Listings 2 and 3)
# --------------------------------------------------------------------------

def init_state(image: np.ndarray, channels: int, dtype) -> np.ndarray:
    """Coarsest-level seed: image in channels [0, n_in), zeros in the hidden ones."""
    d, h, w, n_in = image.shape
    s = np.zeros((d, h, w, channels), dtype=dtype)
    s[..., :n_in] = image
    return s


def upsample_inject(coarse: np.ndarray, factor: Sequence[int], fine_image: np.ndarray,
                    dtype) -> np.ndarray:
    """Nearest-neighbour upsampling of the whole state by integer factors,
    S_l[z,y,x,:] = S_{l+1}[z // fz, y // fy, x // fx, :], followed by
    S_l[..., :n_in] = I_l (the level's image is re-injected)."""
    fz, fy, fx = factor
    d, h, w, n_in = fine_image.shape
    zi = np.arange(d) // fz
    yi = np.arange(h) // fy
    xi = np.arange(w) // fx
    fine = coarse[zi[:, None, None], yi[None, :, None], xi[None, None, :], :].astype(dtype)
    fine[..., :n_in] = fine_image
    return fine


# --------------------------------------------------------------------------
# stochastic fire mask (Sec. 3.1 asynchronous activation; supplement S3)
# --------------------------------------------------------------------------

def fire_threshold(fire_rate: float) -> int:
    """A cell fires iff its 32-bit draw u satisfies u < T, T = floor(p * 2^32)
    with p the single-precision fire rate, capped at 2^32 (p = 1 fires always,
    p = 0 never)."""
    p = float(np.float32(fire_rate))
    if not (0.0 <= p <= 1.0):
        raise ValueError("fire rate must lie in [0, 1]")
    return min(1 << 32, int(np.floor(p * 4294967296.0)))


def fire_bits(seed: int, level: int, step: int, idx: np.ndarray, fire_rate: float,
              batch: int = 0) -> np.ndarray:
    """Fire bit of each cell with canonical linear index ``idx``
    (idx = (z*H + y)*W + x at its level).  Philox4x64-10 with counter
    (idx >> 3, step, level, batch) and key (seed, 0) gives four 64-bit words
    for a block of 8 consecutive cells; cell idx takes word (idx >> 1) & 3 and,
    within it, the upper 32 bits when idx is odd, the lower 32 bits when even.
    ``batch`` is the image's index in a batch (0 for a single image)."""
    idx = np.asarray(idx, dtype=np.uint64)
    octs, where = np.unique(idx >> np.uint64(3), return_inverse=True)
    words = np.stack(philox4x64((octs, np.uint64(step), np.uint64(level), np.uint64(batch)),
                                (np.uint64(seed), np.uint64(0))), axis=-1)   # [octs][4]
    w = words[where.reshape(idx.shape), ((idx >> np.uint64(1)) & np.uint64(3)).astype(np.intp)]
    odd = (idx & np.uint64(1)) == np.uint64(1)
    draw = np.where(odd, w >> np.uint64(32), w & np.uint64(0xFFFFFFFF))
    return draw < np.uint64(fire_threshold(fire_rate))


def fire_mask(seed: int, level: int, step: int, extent: Sequence[int], fire_rate: float,
              batch: int = 0) -> np.ndarray:
    """Fire bits of a whole level, shape [D][H][W] (bool)."""
    d, h, w = extent
    idx = np.arange(d * h * w, dtype=np.uint64)
    return fire_bits(seed, level, step, idx, fire_rate, batch).reshape(d, h, w)


# --------------------------------------------------------------------------
# one NCA step (Sec. 3.1; supplement S3, Listing 1)
# --------------------------------------------------------------------------

def tap_offsets(ndim: int):
    """Neighbourhood offsets (dz, dy, dx) in the order the kernel taps are
    stored: row-major over dz, dy, dx in {-1, 0, 1} (dz = 0 only, for 2D)."""
    zs = (-1, 0, 1) if ndim == 3 else (0,)
    return [(dz, dy, dx) for dz in zs for dy in (-1, 0, 1) for dx in (-1, 0, 1)]


def perceive(state64: np.ndarray, conv_w: np.ndarray, conv_b: np.ndarray, ndim: int) -> np.ndarray:
    """Depthwise perception with zero padding (cross-correlation):
    P[p, c] = b[c] + sum_o K[c, o] * S[p + o, c], S = 0 outside the array."""
    d, h, w, c = state64.shape
    pz = 1 if ndim == 3 else 0
    padded = np.pad(state64, ((pz, pz), (1, 1), (1, 1), (0, 0)))
    out = np.broadcast_to(conv_b.astype(np.float64), state64.shape).copy()
    kw = conv_w.astype(np.float64)
    term = np.empty_like(out)
    for t, (dz, dy, dx) in enumerate(tap_offsets(ndim)):
        nb = padded[pz + dz: pz + dz + d, 1 + dy: 1 + dy + h, 1 + dx: 1 + dx + w, :]
        np.multiply(nb, kw[:, t], out=term)
        out += term
    return out


def update(state64: np.ndarray, percept: np.ndarray, w1, b1, w2) -> np.ndarray:
    """Per-cell MLP on f = [S, P]: u = W2 ReLU(W1 f + b1) (no second bias)."""
    shape = state64.shape
    c = shape[-1]
    f = np.concatenate([state64, percept], axis=-1).reshape(-1, 2 * c)
    hid = f @ w1.astype(np.float64).T
    hid += b1.astype(np.float64)
    np.maximum(hid, 0.0, out=hid)
    u = hid @ w2.astype(np.float64).T
    return u.reshape(shape)


def linear_index(origin: Sequence[int], shape: Sequence[int], grid: Sequence[int]) -> np.ndarray:
    """Canonical index (z*H + y)*W + x of every cell of a window with global
    ``origin`` and ``shape`` inside a level of extent ``grid``."""
    z = np.arange(origin[0], origin[0] + shape[0], dtype=np.int64)
    y = np.arange(origin[1], origin[1] + shape[1], dtype=np.int64)
    x = np.arange(origin[2], origin[2] + shape[2], dtype=np.int64)
    return ((z[:, None, None] * grid[1] + y[None, :, None]) * grid[2] + x[None, None, :])


def nca_step(state: np.ndarray, weights, n_in: int, ndim: int, level: int, step: int,
             seed: int, fire_rate: float, dtype, origin=(0, 0, 0), grid=None,
             batch: int = 0) -> np.ndarray:
    """One synchronous NCA step of every cell of ``state`` (out of place).

    ``state`` covers the window [origin, origin + shape) of a level of extent
    ``grid`` (default: the whole level).  Cells outside the window are taken as
    zero, which is exact at the level's border; in a window, border cells that
    are not at the level's border come out wrong and the caller discards them.
    """
    grid = tuple(state.shape[:3]) if grid is None else tuple(grid)
    s = state.astype(np.float64)
    p = perceive(s, weights.conv_w, weights.conv_b, ndim)
    u = update(s, p, weights.w1, weights.b1, weights.w2)
    idx = linear_index(origin, state.shape[:3], grid)
    m = fire_bits(seed, level, step, idx, fire_rate, batch).astype(np.float64)
    new = s.copy()
    new[..., n_in:] = s[..., n_in:] + m[..., None] * u[..., n_in:]
    return to_storage(new, dtype)


def run_level(state: np.ndarray, weights, n_in: int, ndim: int, level: int, steps: int,
              seed: int, fire_rate: float, dtype, batch: int = 0) -> np.ndarray:
    """``steps`` consecutive steps t = 0 .. steps-1 of one level."""
    for t in range(steps):
        state = nca_step(state, weights, n_in, ndim, level, t, seed, fire_rate, dtype,
                         batch=batch)
    return state


# --------------------------------------------------------------------------
# readout and whole inference
# --------------------------------------------------------------------------

def first_level_steps(alpha0: float, coarsest: Sequence[int]) -> int:
    """Steps of the first (coarsest) level, alpha0 * max(H, W, D) of that
    level's extent (supplement S10 ablation; rounded down, a reading: the
    paper does not state the rounding)."""
    return int(np.floor(np.float64(np.float32(alpha0)) * max(int(v) for v in coarsest)))


def readout(state: np.ndarray) -> np.ndarray:
    """Two-class segmentation: 1 where the last channel is strictly greater than
    the one before it, else 0 (ties, and any NaN, give 0)."""
    return (state[..., -1] > state[..., -2]).astype(np.uint8)


def readout_classes(state: np.ndarray, classes: int) -> np.ndarray:
    """K-class segmentation from the last K channels (the paper's surgery data
    has several classes, Sec. 4): the index k in [0, K) of the largest of
    state[..., C-K+k], scanning k upwards and moving only on a strictly greater
    value, so ties go to the lower index and a NaN is never chosen over an
    earlier channel.  K = 2 is ``readout``."""
    c = state.shape[-1]
    assert 2 <= classes <= c
    s = state[..., c - classes:]
    best = np.zeros(state.shape[:-1], dtype=np.intp)
    best_val = s[..., 0]
    for k in range(1, classes):
        up = s[..., k] > best_val
        best = np.where(up, k, best)
        best_val = np.where(up, s[..., k], best_val)
    return best.astype(np.uint8)


@dataclass
class InferLog:
    max_abs_per_level: List[float]


def infer(image: np.ndarray, weights: Sequence, *, ndim: int, n_in: int, channels: int,
          factors: Sequence[Sequence[int]], steps: Sequence[int], fire_rate: float,
          seed: int, dtype, log: Optional[InferLog] = None, batch: int = 0):
    """Full OctreeNCA inference: pyramid, coarsest seed, then for every level
    from coarsest to finest an upsample+inject (except the coarsest) followed
    by that level's steps with that level's weights.  Returns (state, seg) of
    the finest level.  ``batch`` is the image's index in a batch: it only
    enters the fire-mask counter."""
    levels = len(steps)
    assert len(weights) == levels and len(factors) == levels - 1
    pyr = build_pyramid(image, factors, dtype)
    state = init_state(pyr[-1], channels, dtype)
    for lvl in range(levels - 1, -1, -1):
        if lvl < levels - 1:
            state = upsample_inject(state, factors[lvl], pyr[lvl], dtype)
        state = run_level(state, weights[lvl], n_in, ndim, lvl, steps[lvl], seed, fire_rate, dtype,
                          batch=batch)
        if log is not None:
            log.max_abs_per_level.append(float(np.max(np.abs(state.astype(np.float64)))))
    return state, readout(state)


# --------------------------------------------------------------------------
# light-cone windows: exact final values on a small box of a huge level
# --------------------------------------------------------------------------

def _clip(box, grid):
    return tuple((max(0, a), min(n, b)) for (a, b), n in zip(box, grid))


def _dilate(box, r, ndim, grid):
    rz = r if ndim == 3 else 0
    rs = (rz, r, r)
    return _clip(tuple((a - k, b + k) for (a, b), k in zip(box, rs)), grid)


def _parent(box, f):
    return tuple((a // k, (b - 1) // k + 1) for (a, b), k in zip(box, f))


def _shape(box):
    return tuple(b - a for a, b in box)


def _crop(arr, outer, inner):
    sl = tuple(slice(i0 - o0, i1 - o0) for (o0, _), (i0, i1) in zip(outer, inner))
    return arr[sl]


def _image_on_box(image, factors, lvl, box, dtype):
    """I_lvl on ``box``, pooled level by level from the finest image exactly as
    ``build_pyramid`` does, but only over the box's footprint."""
    cum = [1, 1, 1]
    for f in factors[:lvl]:
        cum = [a * b for a, b in zip(cum, f)]
    fine_box = tuple((a * k, b * k) for (a, b), k in zip(box, cum))
    sub = image[fine_box[0][0]:fine_box[0][1], fine_box[1][0]:fine_box[1][1],
                fine_box[2][0]:fine_box[2][1]]
    sub = np.asarray(sub, dtype=dtype)
    for f in factors[:lvl]:
        sub = pool(sub, f, dtype)
    return sub


def infer_window(image: np.ndarray, weights: Sequence, box: Box, *, ndim: int, n_in: int,
                 channels: int, factors: Sequence[Sequence[int]], steps: Sequence[int],
                 fire_rate: float, seed: int, dtype) -> np.ndarray:
    """Final finest-level state on ``box`` only, exactly equal to
    ``infer(...)[0]`` cropped to ``box``.

    A step moves information by one cell, so the value of a cell after S steps
    depends only on the level's initial state within distance S; the initial
    state of level l depends on I_l there and on the final state of level l+1
    at the parent cells.  This walks those dependency boxes from fine to
    coarse, then runs every level only on its box: each step shrinks the
    correctly computed region by one cell at window sides that are not at the
    level's border.
    """
    levels = len(steps)
    grids = [tuple(image.shape[:3])]
    for f in factors:
        grids.append(tuple(g // k for g, k in zip(grids[-1], f)))
    box = _clip(box, grids[0])
    need_final = [None] * levels
    need_init = [None] * levels
    need_final[0] = box
    for lvl in range(levels):
        need_init[lvl] = _dilate(need_final[lvl], steps[lvl], ndim, grids[lvl])
        if lvl + 1 < levels:
            need_final[lvl + 1] = _parent(need_init[lvl], factors[lvl])

    state = None
    for lvl in range(levels - 1, -1, -1):
        win = need_init[lvl]
        img = _image_on_box(image, factors, lvl, win, dtype)
        if lvl == levels - 1:
            state = init_state(img, channels, dtype)
        else:
            coarse_box = need_final[lvl + 1]
            f = factors[lvl]
            zi = np.arange(win[0][0], win[0][1]) // f[0] - coarse_box[0][0]
            yi = np.arange(win[1][0], win[1][1]) // f[1] - coarse_box[1][0]
            xi = np.arange(win[2][0], win[2][1]) // f[2] - coarse_box[2][0]
            state = state[zi[:, None, None], yi[None, :, None], xi[None, None, :], :].astype(dtype)
            state[..., :n_in] = img
        cur = win
        for t in range(steps[lvl]):
            origin = tuple(a for a, _ in cur)
            new = nca_step(state, weights[lvl], n_in, ndim, lvl, t, seed, fire_rate, dtype,
                           origin=origin, grid=grids[lvl])
            # keep the cells whose neighbourhood lay inside the window or the level
            shrunk = []
            for axis, ((a, b), n) in enumerate(zip(cur, grids[lvl])):
                if axis == 0 and ndim == 2:
                    shrunk.append((a, b))
                    continue
                shrunk.append((a if a == 0 else a + 1, b if b == n else b - 1))
            shrunk = tuple(shrunk)
            state = _crop(new, cur, shrunk)
            cur = shrunk
        target = need_final[lvl]
        state = _crop(state, cur, target)
    return state
