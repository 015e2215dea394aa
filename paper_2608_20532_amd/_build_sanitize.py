"""Host-sanitizer builds for the CPU test job (AddressSanitizer + UndefinedBehaviorSanitizer).

The oracle (oracle/f2_oracle.c) and the host half of the HIP library (layout,
workspace sizing, argument validation: everything the CPU tests reach) are
compiled with the sanitizers on their host code; device code is built as usual.
Both use clang's shared sanitizer runtime, which the test job preloads into a
Python process (tests/test_sanitize_host.py).  CPU only: nothing here runs on a GPU.
"""
import glob
import os
import subprocess

from . import _build

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_SO = os.path.join(HERE, "libf2gpu_hostsan.so")
ORACLE_SO = os.path.join(ROOT, "oracle", "liboracle_san.so")
CLANG = "/opt/rocm/llvm/bin/clang"


def runtime() -> str:
    """clang's shared AddressSanitizer runtime (the one the builds below link against)."""
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise FileNotFoundError("clang AddressSanitizer runtime not found under /opt/rocm/llvm")
    return hits[-1]


def build(verbose: bool = False):
    """Build both sanitized libraries in place; returns (library, oracle) paths."""
    san = ["-O1", "-g", "-fno-omit-frame-pointer"]
    oracle_cmd = [CLANG, *san, "-fPIC", "-shared", "-fsanitize=address,undefined", "-shared-libsan",
                  "-o", ORACLE_SO, os.path.join(ROOT, "oracle", "f2_oracle.c")]
    host_only = []
    for flag in ("-fsanitize=address", "-fsanitize=undefined", "-shared-libsan", "-fno-omit-frame-pointer"):
        host_only += ["-Xarch_host", flag]
    flags = [f for f in _build.HIPCC_FLAGS if f != "-O3"]
    lib_cmd = ["hipcc", *flags, "-O1", "-g", *host_only, "-I", os.path.join(ROOT, "include"), _build.SRC,
               "-o", LIB_SO]
    for cmd in (oracle_cmd, lib_cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
    return LIB_SO, ORACLE_SO
