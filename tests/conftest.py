import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def _gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return False


def pytest_collection_modifyitems(config, items):
    if _gpu_available():
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


class _PoisonedTorch:
    """Stands in for the torch module inside the binding during GPU tests:
    outputs the binding allocates are filled with 0xA5 bytes, so a kernel that
    leaves part of an output unwritten fails the comparison instead of passing
    on whatever an earlier identical call left in reused memory."""

    def __init__(self, torch):
        self._torch = torch

    def __getattr__(self, name):
        return getattr(self._torch, name)

    def empty(self, *args, **kwargs):
        t = self._torch.empty(*args, **kwargs)
        if t.is_cuda and t.numel() > 0:
            t.view(self._torch.uint8).fill_(0xA5)
        return t


@pytest.fixture(autouse=True)
def _poison_binding_outputs(request, monkeypatch):
    if "gpu" not in request.keywords or not _gpu_available():
        yield
        return
    import torch

    from paper_2501_04266_amd import _lib
    monkeypatch.setattr(_lib, "torch", _PoisonedTorch(torch))
    yield
