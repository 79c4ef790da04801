"""Host-side sanitizer build of the C ABI (CPU only, no GPU code changes).

``jl_api.cpp`` -- argument checks, caches and launch set-up -- is compiled with
AddressSanitizer and UndefinedBehaviorSanitizer on its host side and linked
with the kernel objects of the normal build into ``_build/libjetlong_san.so``.
The oracle is built the same way into ``_build/libjloracle_san.so``.  Both use
clang's shared sanitizer runtime; a process that loads them must preload it
(``runtime()`` gives its path).  The binding and the oracle load these files
when ``JETLONG_LIB`` / ``JETLONG_ORACLE_LIB`` name them.
"""
from __future__ import annotations

import glob
import os
import subprocess

from . import build as _b

LLVM = "/opt/rocm/lib/llvm"
CLANG = os.path.join(LLVM, "bin", "clang")
CLANGXX = os.path.join(LLVM, "bin", "clang++")
SAN_LIB = os.path.join(_b.BUILD, "libjetlong_san.so")
SAN_ORACLE = os.path.join(_b.BUILD, "libjloracle_san.so")
ORACLE_SRC = os.path.join(_b.ROOT, "oracle", "jl_oracle.c")
# host compiler pass only: device code is built exactly as in the normal library
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer", "-Xarch_host", "-shared-libsan"]
LINK_SAN = ["-fsanitize=address,undefined", "-shared-libsan"]


def runtime() -> str:
    """Path of clang's shared ASan runtime (UBSan is part of it)."""
    hits = sorted(glob.glob(os.path.join(LLVM, "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    if not hits:
        raise FileNotFoundError("clang's shared ASan runtime is not installed")
    return hits[-1]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("failed:\n%s\n%s" % (" ".join(cmd), res.stderr))


def build() -> tuple:
    """Build both sanitized libraries; returns (libjetlong_san, libjloracle_san)."""
    kernels = [os.path.join(_b.BUILD, os.path.splitext(s)[0] + ".o")
               for s in _b.SOURCES if s.endswith(".hip")]
    if not all(os.path.exists(o) for o in kernels):
        _b.build()
    api_o = os.path.join(_b.BUILD, "jl_api_san.o")
    _run([_b.HIPCC] + _b.FLAGS + HOST_SAN + ["-g", "-x", "hip", "-c",
                                             os.path.join(_b.CSRC, "jl_api.cpp"), "-o", api_o])
    _run([CLANGXX, "-shared", "-fPIC"] + LINK_SAN + kernels + [api_o, "-L/opt/rocm/lib",
         "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64", "-o", SAN_LIB])
    _run([CLANG, "-O1", "-g", "-fPIC", "-shared", "-std=c11", "-fno-omit-frame-pointer"] +
         LINK_SAN + ["-fno-sanitize-recover=undefined", ORACLE_SRC, "-o", SAN_ORACLE, "-lm"])
    return SAN_LIB, SAN_ORACLE


if __name__ == "__main__":
    print(build())
