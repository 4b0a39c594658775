import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: oracle runs of more than a few seconds")


def pytest_collection_modifyitems(config, items):
    # GPU tests are skipped (not failed) where no GPU is visible, so that
    # `-m "not gpu"` and a plain run on a CPU-only host both stay green.
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(skip)


@pytest.fixture(autouse=True)
def sentinel_buffers(request, monkeypatch):
    """In GPU tests every output and workspace the binding allocates starts as NaN
    (bytes 0xFF: a NaN in bf16 and in fp32), so an element the library fails to write
    cannot pass a comparison by holding a previous run's result that the caching
    allocator handed back."""
    if "gpu" not in request.keywords:
        yield
        return
    import torch
    import paper_2607_17644_amd.binding as B

    new0, ws0 = B._new, B._workspace

    def new(p, name, dtype, device):
        t = new0(p, name, dtype, device)
        t.view(torch.uint8).fill_(0xFF) if t.numel() else None
        return t

    def workspace(p, op, ws, device):
        fresh = ws is None
        ws = ws0(p, op, ws, device)
        if fresh:
            ws.fill_(0xFF)
        return ws

    monkeypatch.setattr(B, "_new", new)
    monkeypatch.setattr(B, "_workspace", workspace)
    yield
