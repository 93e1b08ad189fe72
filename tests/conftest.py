"""Shared test setup: the ``gpu`` marker, the import path, and a record of
each GPU test's worst errors (parity_records.jsonl, one JSON line per test)."""

import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP path")


@pytest.hookimpl(hookwrapper=True)
def pytest_runtest_makereport(item, call):
    outcome = yield
    rep = outcome.get_result()
    if rep.when == "call":
        item._ra_outcome = rep.outcome


@pytest.fixture(autouse=True)
def _parity_record(request):
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    import gpu_harness
    gpu_harness.reset_record()
    yield
    gpu_harness.write_record(request.node.nodeid,
                             getattr(request.node, "_ra_outcome", "unknown"))
