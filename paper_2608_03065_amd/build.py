"""Build libpsc.so in-tree: host construction and persistence (g++, zlib) +
gfx950 device code (hipcc); and libpsc_probe.so, a measurement aid."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libpsc.so")
PROBE_LIB = os.path.join(HERE, "libpsc_probe.so")
BUILD_DIR = os.path.join(HERE, "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # never let the compiler form packed-fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {cmd[0]} ({r.returncode})")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    host_obj = os.path.join(BUILD_DIR, "psc_build.o")
    dev_obj = os.path.join(BUILD_DIR, "psc_device.o")
    store_obj = os.path.join(BUILD_DIR, "psc_store.o")
    gram_obj = os.path.join(BUILD_DIR, "psc_grammar.o")
    _run(["g++", *HOST_FLAGS, f"-I{ROCM}/include", "-c", os.path.join(CSRC, "psc_build.cpp"), "-o", host_obj])
    _run(["g++", *HOST_FLAGS, f"-I{ROCM}/include", "-c", os.path.join(CSRC, "psc_store.cpp"), "-o", store_obj])
    _run(["g++", *HOST_FLAGS, f"-I{ROCM}/include", "-c", os.path.join(CSRC, "psc_grammar.cpp"), "-o", gram_obj])
    _run([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, "psc_device.hip"), "-o", dev_obj])
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", host_obj, store_obj, gram_obj, dev_obj, "-lz", "-o", tmp])
    os.replace(tmp, LIB)
    # the measurement aid beside it (dependent-load latency; bench.py --latency-probe)
    tmp = PROBE_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", os.path.join(CSRC, "psc_probe.hip"), "-o", tmp])
    os.replace(tmp, PROBE_LIB)
    if verbose:
        print("built", LIB, PROBE_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
