import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
GOLDEN = os.path.join(ROOT, "tests", "golden")
if GOLDEN not in sys.path:
    sys.path.insert(0, GOLDEN)

_MARGINS = pytest.StashKey()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def gpu_available() -> bool:
    try:
        import torch
        return bool(torch.cuda.is_available())
    except Exception:
        return False


@pytest.fixture(scope="session")
def lib():
    """The product library, loaded through its binding (fails loudly if unbuilt)."""
    import paper_2607_16074_amd as jn
    return jn


@pytest.fixture
def margin(request):
    """Record a measured error next to its bar; the session prints every
    record at its end, so the worst errors land in the run's output."""
    store = request.config.stash.setdefault(_MARGINS, [])

    def rec(what: str, value: float, bar: float):
        store.append((request.node.name, what, float(value), float(bar)))
    return rec


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    store = config.stash.get(_MARGINS, [])
    if not store:
        return
    tr = terminalreporter
    tr.write_line("worst measured errors (test | quantity | value / bar):")
    for name, what, value, bar in store:
        tr.write_line(f"  {name} | {what} | {value:.2e} / {bar:.2g}")
