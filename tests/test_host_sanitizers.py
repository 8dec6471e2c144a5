"""The library's host code under AddressSanitizer and UBSan (CPU only).

tests/c_abi/kvc_host_checks drives every entry point's validation and the
host work behind it (layout checks, plan images for up to 2^31 - 128 rows,
staging copy lists) over 600 seeded random layouts and the edge cases of the
row and position limits, against a build of the library whose host code is
instrumented.  Its device addresses are fake, so it runs only where no GPU
is present (it stops at the device check there).
"""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_host_code_under_sanitizers():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present: the checks pass fake device addresses")
    import importlib.util
    spec = importlib.util.spec_from_file_location("kvc_build_host_checks",
                                                  os.path.join(HERE, "c_abi", "build_host_checks.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    exe = mod.build(force=False)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr[-4000:]
    assert "host checks ok" in r.stdout
