import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


_CAPMAN = None


def pytest_configure(config):
    global _CAPMAN
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    _CAPMAN = config.pluginmanager.getplugin("capturemanager")


def announce(msg: str) -> None:
    """Write msg to the process's real stderr, past pytest's fd-level capture, so that a case
    that ends the process is still named in what it printed."""
    if _CAPMAN is not None:
        with _CAPMAN.global_and_fixture_disabled():
            sys.stderr.write(msg + "\n")
            sys.stderr.flush()
    else:
        sys.__stderr__.write(msg + "\n")
        sys.__stderr__.flush()


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle


@pytest.fixture(autouse=True)
def _announce_gpu_case(request):
    """Name every GPU test on the real stderr (not captured) before it touches the device."""
    if request.node.get_closest_marker("gpu") is not None:
        announce(f"[gpu case] {request.node.nodeid}")
    yield


def pytest_collection_modifyitems(config, items):
    """GPU tests are skipped with a reason when no GPU is visible (never silently passed)."""
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if item.get_closest_marker("gpu") is not None:
            item.add_marker(skip)
