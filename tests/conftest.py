import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case at a full workload size")


def flush_print(*args):
    print(*args, flush=True)


@pytest.fixture(scope="session")
def gpu():
    """The built HIP library on cuda:0; GPU tests fail loudly without it.

    Every buffer the binding allocates for the library to write (outputs,
    gradients, saved activations, workspace, decode slots) starts as NaN, so
    an element a kernel misses fails the comparison."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")
    from paper_2608_23463_amd import binding
    binding.load()  # raises if the shared library is missing
    binding.set_poison(True)
    return binding
