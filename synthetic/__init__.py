"""Synthetic workloads (shapes, seeds) and their seeded input/weight generators."""
from .configs import (Workload, WORKLOADS, TINY_2D, MEDIUM_2D, PATHOLOGY_184MP,
                      VOLUME_3D, VIDEO_2DT, scaled)
from .generators import LevelWeights, make_weights, make_image, storage_dtype

__all__ = ["Workload", "WORKLOADS", "TINY_2D", "MEDIUM_2D", "PATHOLOGY_184MP", "VOLUME_3D",
           "VIDEO_2DT", "scaled", "LevelWeights", "make_weights", "make_image", "storage_dtype"]
