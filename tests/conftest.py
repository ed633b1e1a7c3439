import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


def _gpu_selected(config):
    expr = config.getoption("markexpr") or ""
    return "gpu" in expr and "not gpu" not in expr


def _status_line(config, text):
    tr = config.pluginmanager.get_plugin("terminalreporter")
    if tr is not None:
        tr.write_line(text)
        tr.flush()


def pytest_sessionstart(session):
    # In quiet mode a GPU run is otherwise silent until its first test ends,
    # and the first torch import on a freshly started machine is slow.
    if _gpu_selected(session.config):
        _status_line(session.config, "GPU suite: collecting tests")


def pytest_collection_finish(session):
    if _gpu_selected(session.config):
        _status_line(session.config, f"GPU suite: {len(session.items)} tests selected")


@pytest.fixture(autouse=True)
def _progress_lines(request, capsys):
    """GPU tests print a line per step and per oracle prefill; route those
    lines past output capture (see gpu_helpers.log)."""
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    import gpu_helpers
    gpu_helpers._PROGRESS_SINK = capsys
    try:
        yield
    finally:
        gpu_helpers._PROGRESS_SINK = None
