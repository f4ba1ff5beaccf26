import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


_CONFIG = None


def pytest_configure(config):
    global _CONFIG
    _CONFIG = config
    config.addinivalue_line("markers", "gpu: needs an MI355X (HIP device) and the built libmetro.so")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


def progress(*args):
    """Print a line to the real stdout even while pytest captures test output,
    so that a test running for minutes (the full-depth oracle) shows progress
    under -q as well."""
    msg = " ".join(str(a) for a in args)
    capman = _CONFIG.pluginmanager.getplugin("capturemanager") if _CONFIG is not None else None
    if capman is None:
        print(msg, flush=True)
        return
    with capman.global_and_fixture_disabled():
        print(msg, flush=True)


@pytest.fixture(scope="session")
def repo_root():
    return ROOT
