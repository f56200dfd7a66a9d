"""Shared pytest configuration.

Markers: ``gpu`` marks tests that need an MI355X (they call the HIP library
through its C ABI).  Everything else runs on the CPU.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Environment settings that serialise the runtime would hide ordering faults:
# a test of stream ordering is meaningless under them.
SERIALISING_ENV = ("AMD_SERIALIZE_KERNEL", "AMD_SERIALIZE_COPY", "HIP_LAUNCH_BLOCKING",
                   "CUDA_LAUNCH_BLOCKING")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU (HIP library through the C ABI)")


@pytest.fixture(autouse=True)
def _gpu_preconditions(request):
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    bad = [k for k in SERIALISING_ENV if os.environ.get(k, "0") not in ("", "0")]
    if bad:
        pytest.fail(f"serialising environment variables set ({bad}); ordering tests would be vacuous")
    import torch  # noqa: F401  (the HIP runtime must come from torch's process image)
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    yield
