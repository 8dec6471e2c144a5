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


def ensure_c_demo():
    """Build the plain-C client tests/c_abi/kvc_c_demo (gcc) if it is missing
    or older than its source or the library."""
    import subprocess
    lib = ensure_library()
    d = os.path.join(ROOT, "tests", "c_abi")
    src, exe = os.path.join(d, "kvc_c_demo.c"), os.path.join(d, "kvc_c_demo")
    if os.path.exists(exe) and os.path.getmtime(exe) >= max(os.path.getmtime(src), os.path.getmtime(lib)):
        return exe
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), src, "-L" + os.path.dirname(lib), "-lkvc", "-L/opt/rocm/lib",
           "-lamdhip64", "-Wl,-rpath,$ORIGIN/../../paper_2609_09768_amd", "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


@pytest.fixture(scope="session")
def c_demo():
    return ensure_c_demo()


@pytest.fixture(scope="session")
def K():
    ensure_library()
    import paper_2609_09768_amd as K
    return K
