import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
for p in (ROOT, os.path.join(ROOT, "tests")):
    if p not in sys.path:
        sys.path.insert(0, p)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_collection_finish(session):
    """Start the oracle runs the selected full-size raster tests need, in
    worker processes, before any test touches the GPU (they take about a
    minute each and overlap the other GPU tests).  session.items holds the
    selected tests only."""
    if session.config.getoption("collectonly", default=False):
        return
    owner, keys = None, []
    for item in session.items:
        mod = getattr(item, "module", None)
        if mod is not None and hasattr(mod, "JOBS_FOR") and item.get_closest_marker("gpu"):
            owner = mod
            keys += [k for k in mod.JOBS_FOR(item.nodeid) if k not in keys]
    if keys:
        owner.start_oracle_jobs(keys)
