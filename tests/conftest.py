import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_addoption(parser):
    parser.addoption("--dion2-lib", default=None,
                     help="load this build of libdion2.so (e.g. the host-sanitized one) instead of the package's")


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) HIP device; parity tests proper")
    path = config.getoption("--dion2-lib")
    if path:
        from paper_2512_16928_amd import binding
        binding.load(os.path.abspath(path))


@pytest.fixture(scope="session")
def hip_device():
    """The HIP device for GPU tests; fails (does not skip) when the library or
    the device is missing, so a GPU run can never pass without native code."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("gpu-marked test run without a visible HIP device")
    from paper_2512_16928_amd import binding
    binding.load()  # raises if libdion2.so is missing
    return torch.device("cuda:0")
