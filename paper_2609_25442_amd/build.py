"""Build libwb.so in-tree: host C++ with g++, gfx950 kernels with hipcc.

Run as ``python paper_2609_25442_amd/build.py`` (by path: importing the package
needs the library). Always recompiles.
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libwb.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HOST_SOURCES = ["api.cpp", "layout.cpp", "plan.cpp", "probe.cpp"]
DEVICE_SOURCES = ["kernels.hip", "probe.hip", "noalloc.hip"]
# no packed fp32 instructions: hipcc would otherwise form v_pk_*_f32 by itself
DEVICE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I" + os.path.join(ROCM, "include")]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {cmd[0]} {cmd[-1]}")
    return r


def build(verbose: bool = False, out: str = OUT, defines=()) -> str:
    """Compile and link libwb.so at ``out``; ``defines`` are extra -D flags for
    the host and device sources (tuning knobs such as WB_CHUNK_PER_LANE)."""
    bdir = os.path.join(ROOT, "_build", os.path.basename(out) + ".d")
    os.makedirs(bdir, exist_ok=True)
    objs = []
    for s in HOST_SOURCES:
        o = os.path.join(bdir, s + ".o")
        _run(["g++", *HOST_FLAGS, *["-D" + d for d in defines], "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    for s in DEVICE_SOURCES:
        o = os.path.join(bdir, s + ".o")
        _run([HIPCC, *DEVICE_FLAGS, *["-D" + d for d in defines], "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    tmp = out + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, out)
    if verbose:
        print("built", out)
    return out


if __name__ == "__main__":
    build(verbose=True)
