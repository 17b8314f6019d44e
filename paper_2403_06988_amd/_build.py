"""Compile libdv.so (the HIP kernels and the C ABI of include/dv.h) and
libdv_probes.so (the roofline probes of include/dv_probes.h, measurement
only) for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = ["dv_api.hip", "dv_align.hip", "dv_step.hip", "dv_spec.hip", "dv_sample.hip"]
PROBE_SOURCES = ["dv_probes.hip"]
LIB = os.path.join(HERE, "libdv.so")
PROBE_LIB = os.path.join(HERE, "libdv_probes.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function", "-fvisibility=hidden",
    # packed fp32 ops stay off: the compiler must not form v_pk_*_f32 by itself
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(out: str, sources, verbose: bool) -> str:
    cmd = [HIPCC, *FLAGS, "-o", out + ".tmp", *[os.path.join(CSRC, s) for s in sources]]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def build(verbose: bool = False) -> str:
    """Both libraries; returns the path of libdv.so."""
    _compile(PROBE_LIB, PROBE_SOURCES, verbose)
    return _compile(LIB, SOURCES, verbose)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
