"""Host-only sanitizer build of the C ABI (AddressSanitizer + UBSan).

The host code (``csrc/digest_host.cpp``: argument checks, the partition's
index maps, workspace layout, launch planning) is compiled by g++ with the
sanitizers and linked with the ordinary gfx950 kernel object into
``_build/libdigest_host_sanitized.so``.  No GPU code is built with a
sanitizer.  The library is for CPU-side runs only (creating, querying and
exporting partitions, every error path); load it with the sanitizer runtimes
preloaded and ``DIGEST_LIBRARY`` pointing at it, e.g.

    LD_PRELOAD="$(g++ -print-file-name=libasan.so) $(g++ -print-file-name=libubsan.so)" \\
    ASAN_OPTIONS=detect_leaks=0 DIGEST_LIBRARY=<path> python -m pytest tests/test_abi_cpu.py

    python -m paper_2206_00057_amd.build_sanitized      # prints the library path
"""
from __future__ import annotations

import os
import subprocess
import sys

from . import build as B

SANITIZERS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer"]
LIB = os.path.join(B.BUILD, "libdigest_host_sanitized.so")


def runtime_preload() -> str:
    """The LD_PRELOAD value that loads g++'s sanitizer runtimes."""
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        path = subprocess.run(["g++", f"-print-file-name={name}"], stdout=subprocess.PIPE,
                              text=True, check=True).stdout.strip()
        libs.append(path)
    return " ".join(libs)


def build(verbose: bool = False) -> str:
    os.makedirs(B.BUILD, exist_ok=True)
    kern_o = os.path.join(B.BUILD, "digest_kernels.o")
    if not os.path.exists(kern_o):
        B.build(verbose)
    host_o = os.path.join(B.BUILD, "digest_host_sanitized.o")
    flags = [f for f in B.CXX_FLAGS if f != "-O2"] + ["-O1", "-g"] + SANITIZERS
    B._run(["g++", *flags, "-c", os.path.join(B.CSRC, "digest_host.cpp"), "-o", host_o],
           verbose)
    tmp = LIB + f".tmp{os.getpid()}"
    B._run(["g++", "-shared", *SANITIZERS, host_o, kern_o, "-o", tmp,
            "-L", os.path.join(B.ROCM, "lib"), "-lamdhip64",
            f"-Wl,-rpath,{os.path.join(B.ROCM, 'lib')}"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
