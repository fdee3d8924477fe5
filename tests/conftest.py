import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TESTS = os.path.dirname(os.path.abspath(__file__))
for p in (ROOT, TESTS):
    if p not in sys.path:
        sys.path.insert(0, p)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def _ensure_library():
    """Load what is built; build only when no library exists yet."""
    from paper_2508_06993_amd.build import LIB_PATH, build
    if not os.path.exists(LIB_PATH):
        build()
    return LIB_PATH


@pytest.fixture(scope="session")
def library_path():
    return _ensure_library()


@pytest.fixture(scope="session")
def gpu():
    """The GPU tests' device.  No GPU (or no library) is an error, not a skip,
    on a machine that runs them: the HIP path must be the one that runs."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this environment")
    _ensure_library()
    import paper_2508_06993_amd as octnca
    octnca.lib()
    torch.cuda.set_device(0)
    return torch.device("cuda", 0)


STEP_KERNELS = ("mfma", "mfma_rows", "mfma_tiles", "mfma_f32", "mfma_bf16x3", "valu")


@pytest.fixture(params=STEP_KERNELS)
def step_kernel(request, monkeypatch):
    """Run a test once per fused-step kernel (the library reads
    OCTREE_NCA_STEP_KERNEL at every launch).  "mfma" is the default kernel:
    scaled fp16 activations with split fp16 weights for fp32 states, fp16
    operands for fp16 states, and for 2D the work layout chosen by level
    size; "mfma_rows" and "mfma_tiles" force the 2D layout (row streaming,
    16 x 32 tiles) so both are covered at test sizes; "mfma_f32" uses fp32 MLP
    operands, "mfma_bf16x3" split-bf16 ones; "valu" is the one-thread-per-cell
    vector kernel."""
    monkeypatch.setenv("OCTREE_NCA_STEP_KERNEL", request.param)
    return request.param
