import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle.attention as O
    return O


@pytest.hookimpl(hookwrapper=True, trylast=True)
def pytest_runtest_call(item):
    """GPU tests print as they go (the case each GPU step runs, and the
    oracle's progress over its pieces), so a long oracle check is never a
    silent minutes-long stretch and a fault still leaves its case named.
    (Innermost wrapper of the call phase: inside the capture plugin's, which
    turns capture on for the phase.)"""
    if item.get_closest_marker("gpu") is None:
        yield
        return
    capman = item.config.pluginmanager.getplugin("capturemanager")
    with capman.global_and_fixture_disabled():
        yield
