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
    """The built library, rebuilt first when it is missing or was built from
    other sources than the tree's (its stamp differs)."""
    from paper_2508_06993_amd.build import LIB_PATH, build, is_current
    if not is_current():
        build()
    return LIB_PATH


@pytest.fixture(scope="session")
def library_path():
    return _ensure_library()


@pytest.fixture(scope="session")
def gpu():
    """The GPU tests' device.  Where no GPU is visible (a CPU-only machine)
    the GPU tests are skipped; where one is, the library must build and load:
    a failure there is an error, and there is no CPU fallback to pass on."""
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
def step_kernel(request):
    """Run a test once per fused-step kernel; the test passes the name to
    ``Model(kernel=...)``, which sets the step-kernel fields of the C model
    description.  "mfma" is the default kernel: scaled fp16 activations with
    split fp16 weights for fp32 states, fp16 operands for fp16 states, and for
    2D the work layout chosen by level size; "mfma_rows" and "mfma_tiles"
    force the 2D layout (row streaming, 16 x 32 tiles) so both are covered at
    test sizes; "mfma_f32" uses fp32 MLP operands, "mfma_bf16x3" split-bf16
    ones; "valu" is the one-thread-per-cell vector kernel."""
    return request.param
