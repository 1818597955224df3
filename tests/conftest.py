import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _ensure_built():
    """Build the CPU-side libraries only when nothing is built yet."""
    import oracle.build
    import workloads.build
    if not os.path.exists(os.path.join(ROOT, "oracle", "liboracle.so")):
        oracle.build.build()
    if not (os.path.exists(os.path.join(ROOT, "workloads", "libtaot_gen_host.so"))
            and os.path.exists(os.path.join(ROOT, "workloads", "libtaot_gen_dev.so"))):
        workloads.build.build()


_ensure_built()


@pytest.fixture(scope="session")
def gpu():
    """Skip unless a GPU is visible; tests using this are also marked `gpu`."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")
