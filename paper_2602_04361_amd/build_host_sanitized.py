"""Host-sanitized build of the C ABI layer, for CPU-only checks.

The host code of the library (argument validation, geometry tables and their
integer arithmetic in csrc/api.cpp and csrc/geometry.h) is compiled with g++
under AddressSanitizer and UndefinedBehaviorSanitizer and linked with the
regular kernel objects of `python -m paper_2602_04361_amd.build` (no device
code is instrumented) into _build/libsparvar_host_sanitized.so.

Usage: python -m paper_2602_04361_amd.build_host_sanitized
Then run host-only tests against it, e.g.
  LD_PRELOAD=$(g++ -print-file-name=libasan.so) SPARVAR_LIBRARY=_build/libsparvar_host_sanitized.so \\
      python -m pytest tests/test_abi.py
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(BUILD, "libsparvar_host_sanitized.so")
ROCM = "/opt/rocm"
KERNEL_OBJECTS = ["attention.o", "select.o", "decision.o", "cs4a.o", "csla.o", "kv.o", "index.o"]
SAN = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined"]


def asan_runtime() -> str:
    return subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()


def build() -> str:
    objs = [os.path.join(BUILD, o) for o in KERNEL_OBJECTS]
    missing = [o for o in objs if not os.path.exists(o)]
    if missing:
        raise RuntimeError(f"kernel objects missing ({missing[0]}): run `python -m paper_2602_04361_amd.build` first")
    api_o = os.path.join(BUILD, "api_host_sanitized.o")
    compile_cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", *SAN, "-D__HIP_PLATFORM_AMD__",
                   f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
                   "-c", os.path.join(CSRC, "api.cpp"), "-o", api_o]
    link_cmd = ["g++", "-shared", *SAN, api_o, *objs, f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib",
                "-o", LIB]
    for cmd in (compile_cmd, link_cmd):
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return LIB


if __name__ == "__main__":
    try:
        print(build())
    except RuntimeError as e:
        print(e, file=sys.stderr)
        sys.exit(1)
