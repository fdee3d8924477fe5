"""Synthetic workloads (shapes, seeds) and their seeded input/weight generators."""
from .configs import (Workload, WORKLOADS, TINY_2D, MEDIUM_2D, PATHOLOGY_184MP,
                      VOLUME_3D, VIDEO_2DT, PATHOLOGY_TRAIN_320, TRAIN_WORKLOADS, scaled)
from .generators import LevelWeights, make_weights, make_image, make_target, storage_dtype

__all__ = ["Workload", "WORKLOADS", "TINY_2D", "MEDIUM_2D", "PATHOLOGY_184MP", "VOLUME_3D",
           "VIDEO_2DT", "PATHOLOGY_TRAIN_320", "TRAIN_WORKLOADS", "scaled", "LevelWeights",
           "make_weights", "make_image", "make_target", "storage_dtype"]
