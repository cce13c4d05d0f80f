"""Build the sanitizer check of the C ABI's host code (test infrastructure).

The library's host code (mdlstm_api.cpp) is recompiled with AddressSanitizer
and UndefinedBehaviorSanitizer on its host pass only, linked with the kernel
objects of the regular in-tree build into _build/sanitize/libmdlstm_san.so, and
abi_fuzz.c is built against it with the same sanitizers. Needs the regular
build's objects (python -m paper_1902_11208_amd.build).

Usage: python tests/sanitize/build.py
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from paper_1902_11208_amd import build as libbuild  # noqa: E402

OUT = os.path.join(libbuild.BUILD, "sanitize")
LIB = os.path.join(OUT, "libmdlstm_san.so")
EXE = os.path.join(OUT, "abi_fuzz")
CLANG = os.environ.get("CLANG", "/opt/rocm/llvm/bin/clang")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{cmd[0]} failed:\n{r.stdout}\n{r.stderr}")


def build() -> str:
    os.makedirs(OUT, exist_ok=True)
    kernels = [os.path.join(libbuild.BUILD, os.path.splitext(s)[0] + ".o") for s in libbuild.SOURCES
               if s.endswith(".hip")]
    missing = [k for k in kernels if not os.path.exists(k)]
    if missing:
        raise RuntimeError(f"regular build objects missing: {missing}")
    api_o = os.path.join(OUT, "mdlstm_api.o")
    # each sanitizer flag applies to the host pass only (no device code is instrumented)
    host_san = [x for f in SAN for x in ("-Xarch_host", f)]
    _run([libbuild.HIPCC, *libbuild.FLAGS, "-O1", "-g", *host_san, "-x", "hip", "-c",
          os.path.join(libbuild.CSRC, "mdlstm_api.cpp"), "-o", api_o])
    _run([libbuild.HIPCC, f"--offload-arch={libbuild.ARCH}", "-shared", "-fPIC", *host_san, api_o, *kernels,
          "-o", LIB])
    _run([CLANG, "-std=c11", "-O1", "-g", *SAN, "-I", libbuild.INCLUDE, os.path.join(HERE, "abi_fuzz.c"),
          "-o", EXE, LIB, f"-Wl,-rpath,{OUT}"])
    return EXE


if __name__ == "__main__":
    print(build())
