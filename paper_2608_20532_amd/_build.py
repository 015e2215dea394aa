"""Compile the HIP libraries in place (gfx950 only): the product library
libf2gpu.so and the ceiling-probe library libf2probe.so."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "f2gpu.hip")
SO = os.path.join(HERE, "libf2gpu.so")
PROBE_SRC = os.path.join(HERE, "csrc", "f2probe.hip")
PROBE_SO = os.path.join(HERE, "libf2probe.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def _hipcc(src: str, so: str, verbose: bool) -> str:
    tmp = so + ".tmp"
    cmd = ["hipcc", *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), src, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, so)
    return so


def build(verbose: bool = False) -> str:
    _hipcc(PROBE_SRC, PROBE_SO, verbose)
    return _hipcc(SRC, SO, verbose)
