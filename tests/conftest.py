import os
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(REPO, "tests", "golden")
if REPO not in sys.path:
    sys.path.insert(0, REPO)


def _ensure_built():
    """Build the oracle and the HIP library only if nothing is built yet."""
    if not os.path.exists(os.path.join(REPO, "oracle", "liboracle.so")):
        from oracle import build as ob
        ob.build()
    if not os.path.exists(os.path.join(REPO, "paper_1706_06873_amd", "libmec.so")):
        import importlib.util
        spec = importlib.util.spec_from_file_location(
            "_mec_build", os.path.join(REPO, "paper_1706_06873_amd", "build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()


_ensure_built()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle
