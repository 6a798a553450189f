import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP libraries")
    config.addinivalue_line("markers", "slow: full-size workloads (minutes)")


def _ensure_built():
    """Build the CPU-side libraries only if nothing is built yet (the build
    entry point is the place that always rebuilds)."""
    import oracle
    import synth.native as sn

    if not os.path.exists(oracle.LIB):
        oracle.build()
    if not os.path.exists(sn.HOST_LIB):
        sn.build()


_ensure_built()
