"""On-disk cache of generated images (the 184 MP image takes ~25 s to paint).

Files live in $OCTNCA_IMAGE_CACHE (default /tmp/octnca_images) as .npy, keyed
by workload name, extent, kind and seed; they are only a copy of what
``make_image`` returns.
"""
from __future__ import annotations

import os

import numpy as np

from .configs import Workload
from .generators import make_image


def image_cache_path(wl: Workload, seed: int | None = None) -> str:
    seed = wl.seed if seed is None else seed
    root = os.environ.get("OCTNCA_IMAGE_CACHE", "/tmp/octnca_images")
    d, h, w = wl.extent
    return os.path.join(root, f"{wl.image_kind}_{d}x{h}x{w}x{wl.n_in}_{wl.dtype}_s{seed}.npy")


def cached_image(wl: Workload, seed: int | None = None) -> np.ndarray:
    path = image_cache_path(wl, seed)
    if os.path.exists(path):
        return np.load(path, mmap_mode="r")
    img = make_image(wl, wl.seed if seed is None else seed)
    try:
        os.makedirs(os.path.dirname(path), exist_ok=True)
        tmp = f"{path}.{os.getpid()}.tmp"
        with open(tmp, "wb") as f:
            np.save(f, img)
        os.replace(tmp, path)
    except OSError:
        pass
    return img


def cached_image_file(wl: Workload, seed: int | None = None) -> str:
    """Path of the cached .npy image, written first if it is not there."""
    path = image_cache_path(wl, seed)
    if not os.path.exists(path):
        cached_image(wl, seed)
    if not os.path.exists(path):
        raise OSError(f"could not write the image cache {path}")
    return path
