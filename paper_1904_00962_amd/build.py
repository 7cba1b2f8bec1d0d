"""Build the HIP library ``liblamb_mi355x.so`` in-tree for gfx950.

Run ``python -m paper_1904_00962_amd.build``. The kernels are compiled with
FMA contraction off (every fused multiply-add in them is written out), IEEE
division and square root, and packed-fp32 instructions disabled.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "liblamb_mi355x.so")
SOURCES = [os.path.join(CSRC, "lamb_kernels.hip"), os.path.join(CSRC, "lamb_static.hip"),
           os.path.join(CSRC, "lamb_api.cpp")]
HEADERS = [os.path.join(INCLUDE, "lamb_mi355x.h"), os.path.join(CSRC, "lamb_internal.h"),
           os.path.join(CSRC, "lamb_host.h")]
# Measurement only: streams with the kernels' access patterns (bench.py).
PROBE_LIBRARY = os.path.join(PKG, "libstream_probe.so")
PROBE_SOURCES = [os.path.join(CSRC, "stream_probe.hip")]

ARCH = "gfx950"
HIPCC_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math", "-fvisibility=hidden",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


def build(output: str = LIBRARY, verbose: bool = False, defines=()) -> str:
    """Compile the library; ``defines`` are extra -D flags (tuning variants)."""
    tmp = output + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, *["-D" + d for d in defines], "-I", INCLUDE, "-I", CSRC,
           *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s\n%s" % (proc.returncode, proc.stdout, proc.stderr))
    os.replace(tmp, output)
    return output


def build_probe(output: str = PROBE_LIBRARY, verbose: bool = False) -> str:
    """Compile the stream probe used by bench.py (not part of the optimizer)."""
    tmp = output + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", INCLUDE, *PROBE_SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s\n%s" % (proc.returncode, proc.stdout, proc.stderr))
    os.replace(tmp, output)
    return output


def is_stale(output: str = LIBRARY) -> bool:
    if not os.path.exists(output):
        return True
    t = os.path.getmtime(output)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    print(build_probe(verbose="-v" in sys.argv))
