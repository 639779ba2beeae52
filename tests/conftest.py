import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")


@pytest.fixture(autouse=True)
def _announce_gpu_case(request):
    """GPU tests name themselves on stderr before they start (so a run that
    ends early still shows which case was running) and skip without a GPU."""
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    sys.__stderr__.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.__stderr__.flush()
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    yield
