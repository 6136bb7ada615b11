import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    oracle.build(force=False)
    return oracle


@pytest.fixture(params=["1", "2"], ids=["one-launch", "two-launches"])
def fwd_launches(request, monkeypatch):
    """Runs a layer-forward test with both branch launch plans of
    logo_attn_fwd (LOGO_FWD_LAUNCHES, read on every call; it has no effect
    where only the two-launch plan applies)."""
    monkeypatch.setenv("LOGO_FWD_LAUNCHES", request.param)
    return int(request.param)
