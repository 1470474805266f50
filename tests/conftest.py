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
    cbuild = _load_c_build()
    if not os.path.exists(cbuild.EXE):
        cbuild.build_c_tests()
    yield


def _load_c_build():
    """tests/c/build.py (the C-ABI test program's build), loaded by path."""
    import importlib.util

    spec = importlib.util.spec_from_file_location("pulse_c_test_build", os.path.join(ROOT, "tests", "c", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod
