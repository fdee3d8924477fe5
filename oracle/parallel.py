"""Process-parallel drivers of the oracle -- TEST INFRASTRUCTURE ONLY.

They let the GPU tests compare whole grids and many light-cone boxes of the
large workloads within the test time, on the host's cores.  Neither computes
any part of the method itself; both only schedule the oracle's own functions:

* ``infer_banded`` runs ``octree_nca.infer``'s sequence (pyramid, coarsest
  seed, per level upsample + inject and the level's steps, readout) with each
  NCA step of a large level split into horizontal bands of rows.  A worker
  process evaluates ``nca_step`` on its band plus one halo row on each side
  (the window form of ``nca_step``, with the band's global origin so the fire
  bits use the canonical cell index) and keeps the band's own rows: a step
  moves information by one cell, so those rows are exact (Sec. 3.1), and the
  result equals ``infer`` up to the rounding order of the float64 matrix
  products (tested on the CPU).
* ``infer_windows`` evaluates ``octree_nca.infer_window`` on many boxes, one
  box per task.

Workers are started with the "spawn" method (fresh interpreters that never
touch a GPU), use one BLAS thread each, and exchange states through shared
memory that the driver creates and removes.
"""
from __future__ import annotations

import os
from concurrent.futures import ProcessPoolExecutor
from multiprocessing import get_context, shared_memory
from types import SimpleNamespace
from typing import List, Optional, Sequence

import numpy as np

from . import octree_nca as onca

# levels with fewer cells than this run in the calling process
_MIN_PARALLEL_CELLS = 1 << 16


def default_workers() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _plain_weights(weights) -> List[SimpleNamespace]:
    return [SimpleNamespace(**{k: np.asarray(getattr(w, k)) for k in
                               ("conv_w", "conv_b", "w1", "b1", "w2")}) for w in weights]


# --------------------------------------------------------------------------
# worker side
# --------------------------------------------------------------------------

_W: dict = {}


def _limit_blas():
    try:
        from threadpoolctl import threadpool_limits
        _W["blas"] = threadpool_limits(1)
    except Exception:   # pragma: no cover
        pass


def _band_init(shm_names, weights, params):
    _limit_blas()
    _W["shm"] = [shared_memory.SharedMemory(name=n) for n in shm_names]
    _W["weights"] = weights
    _W["p"] = params


def _band_step(task):
    """One NCA step of rows [y0, y1) of the level held in buffer src
    (extent ext), written to the same rows of buffer dst."""
    src, dst, ext, y0, y1, level, step = task
    p = _W["p"]
    d, h, w = ext
    dtype = np.dtype(p["dtype"])
    shape = (d, h, w, p["channels"])
    a = np.ndarray(shape, dtype=dtype, buffer=_W["shm"][src].buf)
    b = np.ndarray(shape, dtype=dtype, buffer=_W["shm"][dst].buf)
    lo, hi = max(0, y0 - 1), min(h, y1 + 1)
    new = onca.nca_step(np.array(a[:, lo:hi]), _W["weights"][level], p["n_in"], p["ndim"], level,
                        step, p["seed"], p["fire_rate"], dtype, origin=(0, lo, 0), grid=ext,
                        batch=p["batch"])
    b[:, y0:y1] = new[:, y0 - lo:y1 - lo]
    return y1 - y0


def _window_init(image_path, weights, params):
    _limit_blas()
    _W["image"] = np.load(image_path, mmap_mode="r")
    _W["weights"] = weights
    _W["p"] = params


def _window_task(box):
    p = _W["p"]
    return onca.infer_window(_W["image"], _W["weights"], box, ndim=p["ndim"], n_in=p["n_in"],
                             channels=p["channels"], factors=p["factors"], steps=p["steps"],
                             fire_rate=p["fire_rate"], seed=p["seed"], dtype=np.dtype(p["dtype"]))


# --------------------------------------------------------------------------
# drivers
# --------------------------------------------------------------------------

def infer_banded(image: np.ndarray, weights: Sequence, *, ndim: int, n_in: int, channels: int,
                 factors, steps: Sequence[int], fire_rate: float, seed: int, dtype,
                 batch: int = 0, workers: Optional[int] = None):
    """``octree_nca.infer`` with the steps of large levels evaluated band by
    band in worker processes.  Returns (state, seg) of the finest level."""
    workers = workers or default_workers()
    dtype = np.dtype(dtype)
    levels = len(steps)
    assert len(weights) == levels and len(factors) == levels - 1
    pyr = onca.build_pyramid(image, factors, dtype)
    state = onca.init_state(pyr[-1], channels, dtype)
    finest = int(np.prod(image.shape[:3]))
    nbytes = finest * channels * dtype.itemsize
    shms = [shared_memory.SharedMemory(create=True, size=nbytes) for _ in range(2)]
    plain = _plain_weights(weights)
    params = dict(dtype=dtype.str, channels=channels, n_in=n_in, ndim=ndim, seed=seed,
                  fire_rate=fire_rate, batch=batch)
    try:
        ctx = get_context("spawn")
        with ProcessPoolExecutor(max_workers=workers, mp_context=ctx, initializer=_band_init,
                                 initargs=([s.name for s in shms], plain, params)) as pool:
            for lvl in range(levels - 1, -1, -1):
                if lvl < levels - 1:
                    state = onca.upsample_inject(state, factors[lvl], pyr[lvl], dtype)
                d, h, w = state.shape[:3]
                if d * h * w < _MIN_PARALLEL_CELLS or steps[lvl] == 0:
                    state = onca.run_level(state, weights[lvl], n_in, ndim, lvl, steps[lvl], seed,
                                           fire_rate, dtype, batch=batch)
                    continue
                views = [np.ndarray(state.shape, dtype=dtype, buffer=s.buf) for s in shms]
                views[0][...] = state
                nb = min(h, 4 * workers)
                edges = [h * i // nb for i in range(nb + 1)]
                cur = 0
                for t in range(steps[lvl]):
                    tasks = [(cur, cur ^ 1, (d, h, w), edges[i], edges[i + 1], lvl, t)
                             for i in range(nb) if edges[i + 1] > edges[i]]
                    done = sum(pool.map(_band_step, tasks))
                    assert done == h
                    cur ^= 1
                state = np.array(views[cur])
                del views
    finally:
        for s in shms:
            s.close()
            s.unlink()
    return state, onca.readout(state)


def infer_windows(image_path: str, weights: Sequence, boxes, *, ndim: int, n_in: int,
                  channels: int, factors, steps: Sequence[int], fire_rate: float, seed: int,
                  dtype, workers: Optional[int] = None) -> List[np.ndarray]:
    """``octree_nca.infer_window`` on each box of ``boxes`` (the image is read
    from the .npy file at ``image_path``, memory-mapped by every worker)."""
    workers = workers or default_workers()
    params = dict(ndim=ndim, n_in=n_in, channels=channels,
                  factors=[tuple(int(v) for v in f) for f in factors],
                  steps=[int(s) for s in steps], fire_rate=fire_rate, seed=seed,
                  dtype=np.dtype(dtype).str)
    ctx = get_context("spawn")
    with ProcessPoolExecutor(max_workers=workers, mp_context=ctx, initializer=_window_init,
                             initargs=(image_path, _plain_weights(weights), params)) as pool:
        return list(pool.map(_window_task, [tuple(tuple(int(v) for v in ax) for ax in b)
                                            for b in boxes]))
