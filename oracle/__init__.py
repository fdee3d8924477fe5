"""CPU oracle for OctreeNCA inference -- TEST INFRASTRUCTURE ONLY.

A plain, slow float64 implementation of what the GPU path computes, written
from the paper (arXiv 2508.06993, Sec. 3.1-3.2 and supplement S3, S6, S7).
Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it.  It shares no code with the HIP library, and the
library never calls it.

Pins (tests that fix it to something other than itself) are listed in each
function's docstring and in tests/test_oracle_*.py.  End-to-end values have no
printed worked example in the paper; they are pinned only through the pinned
parts (brute-force per-cell loops, library routines, invariants).
"""
from .philox import philox4x64, mulhilo64
from .octree_nca import (pool, build_pyramid, init_state, upsample_inject, fire_threshold,
                         fire_bits, fire_mask, tap_offsets, perceive, update, nca_step,
                         run_level, readout, readout_classes, first_level_steps, infer,
                         infer_window, linear_index, to_storage, InferLog)
from .train import (LevelGrads, step_vjp, level_states, level_vjp, upsample_vjp, Tape,
                    train_forward, train_backward, readout_mse)
