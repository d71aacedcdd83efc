import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


import pytest  # noqa: E402


@pytest.fixture(scope="session")
def stream_case():
    """The oracle's offline model of the 32-layer decode stack (built once)."""
    import workloads as wl
    from tests._pipeline import build_stream
    return build_stream(wl.C5_STREAM)
