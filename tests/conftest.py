import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session", autouse=True)
def _built_artifacts():
    """Build what is missing (tests load what is built and build only if nothing is)."""
    from oracle import build as obuild

    if not os.path.exists(obuild.LIB):
        obuild.build_oracle()
    from paper_2609_34555_amd import _build as pbuild

    if not os.path.exists(pbuild.LIB):
        pbuild.build_library()
    yield
