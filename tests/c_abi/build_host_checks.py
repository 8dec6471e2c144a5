"""Builds the host-sanitizer checks (CPU only; no GPU is needed or used).

* paper_2609_09768_amd/libkvc_hostsan.so: the library from the same
  sources, with AddressSanitizer and UndefinedBehaviorSanitizer on its host
  code (validation, plan images, staging copy lists); device code is
  compiled as usual.
* tests/c_abi/kvc_host_checks: the C driver of those checks, built with the
  same sanitizers and linked against that library.

    python tests/c_abi/build_host_checks.py
"""
import importlib.util
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2609_09768_amd")
LIB = os.path.join(PKG, "libkvc_hostsan.so")
SRC = os.path.join(HERE, "kvc_host_checks.c")
EXE = os.path.join(HERE, "kvc_host_checks")

# each sanitizer flag applies to the host pass only
HOST_SANITIZERS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                   "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
DRIVER_SANITIZERS = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
                     "-fno-omit-frame-pointer"]


def _build_lib_module():
    spec = importlib.util.spec_from_file_location("kvc_build_lib", os.path.join(PKG, "build_lib.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("build failed: " + " ".join(cmd[:2]))


def build(force: bool = True) -> str:
    bl = _build_lib_module()
    srcs = [os.path.join(bl.CSRC, s) for s in bl.SOURCES]
    inputs = srcs + [SRC, os.path.join(ROOT, "include", "kvc.h")]
    if not force and os.path.exists(EXE) and os.path.exists(LIB) and \
            os.path.getmtime(EXE) >= max(os.path.getmtime(p) for p in inputs):
        return EXE
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    flags = [f for f in bl.FLAGS if f != "-O3"] + ["-O1", "-g"]
    _run([hipcc, *flags, *HOST_SANITIZERS, "-I", os.path.join(ROOT, "include"), *srcs, "-o", LIB + ".tmp"])
    os.replace(LIB + ".tmp", LIB)
    clang = "/opt/rocm/llvm/bin/clang"
    _run([clang, "-std=c11", "-O1", "-g", "-Wall", "-Wextra", "-Werror", *DRIVER_SANITIZERS,
          "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), SRC,
          "-L" + PKG, "-l:libkvc_hostsan.so", "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,$ORIGIN/../../paper_2609_09768_amd", "-Wl,-rpath,/opt/rocm/lib", "-o", EXE])
    return EXE


if __name__ == "__main__":
    print(build())
