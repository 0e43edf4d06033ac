import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: longer CPU test")
    config.addinivalue_line("markers", "long_oracle: oracle reference computed in the "
                            "background from the start of the session (tests/long_refs.py)")


def pytest_collection_finish(session):
    """Starts the oracle work of the selected long-batch tests before any
    test runs (and before anything touches the GPU): it then overlaps the
    rest of the suite."""
    if session.config.option.collectonly:
        return
    ids = [item.callspec.id for item in session.items
           if item.get_closest_marker("long_oracle") and hasattr(item, "callspec")]
    if not ids:
        return
    try:
        import torch
        if torch.cuda.device_count() == 0:  # does not initialise the GPU
            return
    except ImportError:
        return
    from tests import long_refs
    long_refs.start(ids)


def pytest_sessionfinish(session, exitstatus):
    mod = sys.modules.get("tests.long_refs")
    if mod is not None:
        mod.stop()
