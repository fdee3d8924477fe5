"""Convenience layer over the binding: upload weights, allocate the workspace
and outputs with PyTorch, run ``octree_nca_infer``.  Allocation and marshalling
only; the computation is the library's.
"""
from __future__ import annotations

import warnings
from typing import List, Optional, Sequence

import numpy as np
import torch

from . import Model, octree_nca_infer, octree_nca_workspace_bytes

WEIGHT_FIELDS = ("conv_w", "conv_b", "w1", "b1", "w2")


def upload_weights(levels, device="cuda") -> List[dict]:
    """Per-level weights (objects or dicts holding fp32 numpy arrays in the
    canonical layout) -> list of dicts of contiguous fp32 device tensors."""
    out = []
    for w in levels:
        get = (lambda k: w[k]) if isinstance(w, dict) else (lambda k: getattr(w, k))
        out.append({k: torch.from_numpy(np.ascontiguousarray(get(k), dtype=np.float32))
                    .to(device) for k in WEIGHT_FIELDS})
    return out


def to_device_image(image: np.ndarray, model: Model, device="cuda") -> torch.Tensor:
    """[D][H][W][n_in] numpy image -> contiguous device tensor of the model's storage type."""
    assert image.ndim == 4 and image.shape[-1] == model.n_in
    with warnings.catch_warnings():
        # a read-only (memory-mapped) array is only read by the copy below
        warnings.filterwarnings("ignore", message="The given NumPy array is not writable")
        t = torch.from_numpy(np.ascontiguousarray(image))
    return t.to(device=device, dtype=model.torch_dtype)


class Inference:
    """Buffers for repeated inference of one model on one finest extent."""

    def __init__(self, model: Model, finest: Sequence[int], factors, device="cuda",
                 want_state=True, want_seg=True):
        self.model = model
        self.finest = tuple(int(v) for v in finest)
        self.factors = [tuple(int(v) for v in f) for f in factors]
        ws = octree_nca_workspace_bytes(model, self.finest, self.factors, want_state)
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)
        d, h, w = self.finest
        self.state = (torch.empty((d, h, w, model.channels), dtype=model.torch_dtype,
                                  device=device) if want_state else None)
        self.seg = torch.empty((d, h, w), dtype=torch.uint8, device=device) if want_seg else None

    def __call__(self, image: torch.Tensor, weights, steps, fire_rate: float, seed: int,
                 level_events=None, stream=None):
        octree_nca_infer(self.model, image, self.factors, weights, steps, fire_rate, seed,
                         self.workspace, self.state, self.seg, level_events, stream)
        return self.state, self.seg


def infer(model: Model, image: torch.Tensor, factors, weights, steps, fire_rate: float,
          seed: int, stream=None):
    """One-shot inference; returns (final state, seg) as device tensors."""
    run = Inference(model, image.shape[:3], factors, device=image.device)
    return run(image, weights, steps, fire_rate, seed, stream=stream)
