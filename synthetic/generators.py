"""Seeded synthetic inputs and random-initialised weights for the workloads.

These generators are shared by the GPU path's tests/benchmark and by the
oracle's tests.  They draw random numbers and paint images; they contain no
part of the NCA method (no pooling, no perception, no update rule).

Draw order (documented so that any consumer can regenerate the same data):

* image rng   = numpy.random.default_rng([seed, 0])
* weights rng = numpy.random.default_rng([seed, 1]); for level l = 0..L-1
  (0 = finest) draw conv_w [C][3^ndim], conv_b [C], w1 [H][2C], b1 [H],
  w2 [C][H], each from normal(mean 0, std 0.1), stored as float32.

The paper trains its NCAs; no trained weights are available, so every level
gets random weights of the paper's architecture (Sec. 3.1, supplement S7:
C = 16 state channels, hidden size 64, 3x3(x3) kernels).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np

from .configs import Workload

WEIGHT_STD = 0.1


@dataclass
class LevelWeights:
    conv_w: np.ndarray  # [C][3^ndim] float32, taps row-major over (dz, dy, dx)
    conv_b: np.ndarray  # [C]
    w1: np.ndarray      # [H][2C]; columns 0..C-1 act on the state, C..2C-1 on the perception
    b1: np.ndarray      # [H]
    w2: np.ndarray      # [C][H]; rows < n_in are never used (input channels are not updated)

    def arrays(self):
        return (self.conv_w, self.conv_b, self.w1, self.b1, self.w2)


def make_weights(wl: Workload, seed: int | None = None, std: float = WEIGHT_STD) -> List[LevelWeights]:
    seed = wl.seed if seed is None else seed
    rng = np.random.default_rng([seed, 1])
    c, h, taps = wl.channels, wl.hidden, wl.taps()
    out = []
    for _ in range(wl.levels):
        cw = rng.normal(0.0, std, size=(c, taps)).astype(np.float32)
        cb = rng.normal(0.0, std, size=(c,)).astype(np.float32)
        w1 = rng.normal(0.0, std, size=(h, 2 * c)).astype(np.float32)
        b1 = rng.normal(0.0, std, size=(h,)).astype(np.float32)
        w2 = rng.normal(0.0, std, size=(c, h)).astype(np.float32)
        out.append(LevelWeights(cw, cb, w1, b1, w2))
    return out


def storage_dtype(wl: Workload):
    return np.float16 if wl.dtype == "f16" else np.float32


def make_image(wl: Workload, seed: int | None = None) -> np.ndarray:
    """Finest-level image, shape [D][H][W][n_in], in the workload's storage type."""
    seed = wl.seed if seed is None else seed
    rng = np.random.default_rng([seed, 0])
    d, h, w = wl.extent
    kind = wl.image_kind
    if kind == "uniform":
        img = rng.random((d, h, w, wl.n_in), dtype=np.float32)
    elif kind == "blobs":
        img = _blobs(rng, d, h, w, wl.n_in)
    elif kind == "smoothed_noise":
        img = _smoothed_noise(rng, d, h, w, wl.n_in)
    elif kind == "ellipses":
        img = _ellipses(rng, d, h, w, wl.n_in)
    else:
        raise ValueError(f"unknown image kind {kind!r}")
    return np.ascontiguousarray(img.astype(storage_dtype(wl), copy=False))


def _blobs(rng, d, h, w, n_in, n_blobs=64, noise=0.05):
    """Sum of isotropic Gaussians (centres uniform in the image, sigma uniform in
    [0.01, 0.1] x H, per-channel amplitudes uniform in [0, 1]), built separably
    as Gy^T diag(a_c) Gx, each channel scaled to max 1, then
    x = (1 - noise) * blobs + noise * U[0, 1)."""
    assert d == 1, "blob images are 2D"
    cy = rng.uniform(0, h, n_blobs)
    cx = rng.uniform(0, w, n_blobs)
    sig = rng.uniform(0.01, 0.1, n_blobs) * h
    amp = rng.uniform(0.0, 1.0, (n_in, n_blobs))
    ys = np.arange(h, dtype=np.float64)
    xs = np.arange(w, dtype=np.float64)
    gy = np.exp(-((ys[None, :] - cy[:, None]) ** 2) / (2 * sig[:, None] ** 2)).astype(np.float32)
    gx = np.exp(-((xs[None, :] - cx[:, None]) ** 2) / (2 * sig[:, None] ** 2)).astype(np.float32)
    out = np.empty((1, h, w, n_in), dtype=np.float32)
    for c in range(n_in):
        blob = gy.T @ (amp[c].astype(np.float32)[:, None] * gx)      # [h][w]
        m = float(blob.max())
        blob *= np.float32((1.0 - noise) / m if m > 0 else 0.0)
        blob += np.float32(noise) * rng.random((h, w), dtype=np.float32)
        out[0, :, :, c] = blob
    return out


def _smoothed_noise(rng, d, h, w, n_in, k=5):
    """N(0,1) noise averaged over a k^3 box with zero padding ('same' size)."""
    from scipy.ndimage import uniform_filter
    noise = rng.standard_normal((d, h, w, n_in)).astype(np.float64)
    out = uniform_filter(noise, size=(k, k, k, 1), mode="constant", cval=0.0)
    return out.astype(np.float32)


def _ellipses(rng, t, h, w, n_in, n_ell=12):
    """Moving opaque ellipses over uniform noise.  Semi-axes U[8, 60] px, angle
    U[0, pi), colour U[0,1]^n_in, centre uniform, velocity U[-3, 3] px/frame,
    reflected at the frame edges; painted in a fixed order every frame."""
    a = rng.uniform(8, 60, n_ell)
    b = rng.uniform(8, 60, n_ell)
    ang = rng.uniform(0, np.pi, n_ell)
    col = rng.uniform(0, 1, (n_ell, n_in)).astype(np.float32)
    pos = np.stack([rng.uniform(0, h, n_ell), rng.uniform(0, w, n_ell)], 1)
    vel = rng.uniform(-3, 3, (n_ell, 2))
    out = np.empty((t, h, w, n_in), dtype=np.float16)
    ca, sa = np.cos(ang), np.sin(ang)
    for f in range(t):
        frame = rng.random((h, w, n_in), dtype=np.float32)
        for e in range(n_ell):
            r = max(a[e], b[e])
            y0, y1 = max(0, int(pos[e, 0] - r)), min(h, int(pos[e, 0] + r) + 1)
            x0, x1 = max(0, int(pos[e, 1] - r)), min(w, int(pos[e, 1] + r) + 1)
            if y0 >= y1 or x0 >= x1:
                continue
            yy, xx = np.mgrid[y0:y1, x0:x1]
            dy, dx = yy - pos[e, 0], xx - pos[e, 1]
            u = (dx * ca[e] + dy * sa[e]) / a[e]
            v = (-dx * sa[e] + dy * ca[e]) / b[e]
            inside = u * u + v * v <= 1.0
            frame[y0:y1, x0:x1][inside] = col[e]
        out[f] = frame
        pos += vel
        for ax, lim in ((0, h), (1, w)):
            lo, hi = pos[:, ax] < 0, pos[:, ax] > lim - 1
            pos[lo, ax] = -pos[lo, ax]
            pos[hi, ax] = 2 * (lim - 1) - pos[hi, ax]
            vel[lo | hi, ax] = -vel[lo | hi, ax]
    return out


def make_target(wl: Workload, image: np.ndarray) -> np.ndarray:
    """Synthetic two-class segmentation target [D][H][W][2] (fp32 one-hot) for a
    training workload: class 1 where the image's channel mean exceeds its
    median, class 0 elsewhere.  A label map with the image's structure; no part
    of the method is computed here."""
    m = np.asarray(image, np.float32).mean(axis=-1)
    fg = (m > np.median(m)).astype(np.float32)
    return np.stack([1.0 - fg, fg], axis=-1).astype(np.float32)
