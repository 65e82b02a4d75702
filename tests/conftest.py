import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_sessionstart(session):
    # long oracle builds (the LLaMA-70B shapes) print progress past the capture
    try:
        import gpu_util
    except Exception:
        return
    gpu_util.CAPTURE_MANAGER = session.config.pluginmanager.getplugin("capturemanager")
