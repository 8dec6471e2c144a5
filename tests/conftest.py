import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
for _p in (ROOT, os.path.join(ROOT, "tests")):
    if _p not in sys.path:
        sys.path.insert(0, _p)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size case (minutes of CPU oracle work)")


def ensure_library():
    """Build libkvc.so (hipcc cross-compile) if nothing is built yet."""
    lib = os.path.join(ROOT, "paper_2609_09768_amd", "libkvc.so")
    if not os.path.exists(lib):
        import importlib.util
        spec = importlib.util.spec_from_file_location(
            "kvc_build_lib", os.path.join(ROOT, "paper_2609_09768_amd", "build_lib.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()
    return lib


@pytest.fixture(scope="session")
def K():
    ensure_library()
    import paper_2609_09768_amd as K
    return K
