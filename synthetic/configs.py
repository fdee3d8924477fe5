"""The five OctreeNCA inference workloads, described by shape only.

Each workload is a synthetic stand-in with the shapes of the paper's data
(Sec. 4 datasets; supplement S7 table of octree level resolutions; supplement
S9 table of the largest single-pass inputs).  Nothing here computes any part
of the method: a workload is extents, level count, pooling factors, step
counts, storage type and seeds.

Conventions shared by the GPU path and the oracle:

* level 0 is the finest (original resolution), level L-1 the coarsest;
* ``factors[l]`` is the (fz, fy, fx) pooling factor from level l to level l+1;
* extents are (D, H, W); a 2D workload has D = 1 and ``ndim = 2``;
* a video (2D+t) is a 3D workload with time as the D axis.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

Extent = Tuple[int, int, int]


@dataclass(frozen=True)
class Workload:
    name: str
    ndim: int                      # 2 or 3 (taps 3x3 or 3x3x3)
    extent: Extent                 # finest (D, H, W)
    n_in: int                      # input (image) channels
    factors: Tuple[Extent, ...]    # len = levels - 1, fine -> coarse
    steps: Tuple[int, ...]         # per level, index 0 = finest
    dtype: str = "f32"             # state / image storage: "f32" or "f16"
    channels: int = 16
    hidden: int = 64
    fire_rate: float = 0.5
    seed: int = 0
    image_kind: str = "uniform"    # generator recipe, see generators.py
    description: str = ""

    @property
    def levels(self) -> int:
        return len(self.steps)

    def level_extents(self) -> List[Extent]:
        ext = [tuple(self.extent)]
        for f in self.factors:
            d, h, w = ext[-1]
            if d % f[0] or h % f[1] or w % f[2]:
                raise ValueError(f"{self.name}: extent {ext[-1]} not divisible by {f}")
            ext.append((d // f[0], h // f[1], w // f[2]))
        return ext

    def cells_per_level(self) -> List[int]:
        return [d * h * w for d, h, w in self.level_extents()]

    def cell_steps(self) -> int:
        return sum(c * s for c, s in zip(self.cells_per_level(), self.steps))

    def taps(self) -> int:
        return 3 ** self.ndim

    def params_per_level(self) -> int:
        """conv weights + conv bias + first linear (with bias) + second linear
        producing only the hidden channels, without bias."""
        c, h = self.channels, self.hidden
        return c * self.taps() + c + 2 * c * h + h + h * (c - self.n_in)


def _f2(n):
    return tuple((1, 2, 2) for _ in range(n))


TINY_2D = Workload(
    name="tiny2d", ndim=2, extent=(1, 64, 64), n_in=3, factors=_f2(2),
    steps=(10, 10, 10), image_kind="uniform",
    description="RGB 64x64 U[0,1], 3 levels 64^2 -> 16^2, 10 steps per level")

MEDIUM_2D = Workload(
    name="medium2d", ndim=2, extent=(1, 1024, 1024), n_in=3, factors=_f2(3),
    steps=(20, 20, 20, 20), image_kind="uniform",
    description="RGB 1024x1024 U[0,1], 4 levels 1024^2 -> 128^2, 20 steps per level")

PATHOLOGY_184MP = Workload(
    name="pathology184mp", ndim=2, extent=(1, 11264, 16384), n_in=3, factors=_f2(5),
    steps=(20,) * 6, image_kind="blobs",
    description="RGB 16384x11264 (184.5 MP) smooth blobs + 5% noise, "
                "6 levels 16384x11264 -> 512x352, 20 steps per level")

VOLUME_3D = Workload(
    name="volume3d", ndim=3, extent=(24, 320, 320), n_in=1, factors=_f2(2),
    steps=(20, 20, 20), image_kind="smoothed_noise",
    description="1-channel 320x320x24 N(0,1) smoothed by a 5x5x5 box, "
                "3 levels, 2x2 in-plane pooling, depth kept")

VIDEO_2DT = Workload(
    name="video2dt", ndim=3, extent=(1800, 240, 432), n_in=3,
    factors=((1, 2, 2), (1, 2, 2), (2, 2, 2), (2, 2, 2)),
    steps=(16,) * 5, dtype="f16", image_kind="ellipses",
    description="RGB 240x432 x 1800 frames of moving ellipses on uniform noise, fp16 "
                "state; 5 levels, time pooled at the two coarsest transitions")

WORKLOADS = {w.name: w for w in (TINY_2D, MEDIUM_2D, PATHOLOGY_184MP, VOLUME_3D, VIDEO_2DT)}

# Training workload (the fused training step): the paper trains the pathology
# model on 320 x 320 patches (supplement S7, training details) with the
# five-level octree of its level table; 20 steps per level as the inference
# workloads, fp32 states.
PATHOLOGY_TRAIN_320 = Workload(
    name="pathology_train320", ndim=2, extent=(1, 320, 320), n_in=3, factors=_f2(4),
    steps=(20,) * 5, image_kind="blobs",
    description="RGB 320x320 training patch of smooth blobs + 5% noise, 5 levels "
                "320^2 -> 20^2, 20 steps per level, fp32")

TRAIN_WORKLOADS = {w.name: w for w in (PATHOLOGY_TRAIN_320,)}


def scaled(base: Workload, extent: Extent, steps=None, name=None, **kw) -> Workload:
    """A smaller workload with the same structure (levels, factors, n_in, dtype)
    as ``base`` -- used for parity cases the oracle finishes in seconds."""
    fields = dict(base.__dict__)
    fields.update(kw)
    fields["extent"] = tuple(extent)
    if steps is not None:
        fields["steps"] = tuple(steps)
    fields["name"] = name or f"{base.name}@{'x'.join(map(str, extent))}"
    return Workload(**fields)
