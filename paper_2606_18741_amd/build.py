"""Build libremp_kv.so (KV migration and weight-shard rebuild) and libremp_probe.so (HBM access-pattern
probes, measurement only) for gfx950 in-tree with hipcc.

    python paper_2606_18741_amd/build.py      (a plain script: importing the package needs the library)
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libremp_kv.so")
PROBE_LIB = os.path.join(PKG, "libremp_probe.so")

SOURCES = [os.path.join(CSRC, f) for f in ("plan.cpp", "migrate.hip", "weights_plan.cpp", "weights.hip")]
PROBE_SOURCES = [os.path.join(CSRC, "probe.hip")]   # HBM access-pattern probes (measurement only)

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    "-fvisibility=hidden",
    # never emit packed fp32 instructions (the library has no float math; this keeps it so)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]

# the host-only planner is plain C++; it sees the HIP headers only for hipStream_t / hipEvent_t
CXX_FLAGS = ["-D__HIP_PLATFORM_AMD__"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _link(sources, out: str, verbose: bool) -> str:
    tmp = out + ".tmp"
    rocm_inc = os.path.join(os.path.dirname(os.path.dirname(hipcc())), "include")
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", rocm_inc, "-o", tmp]
    for src in sources:
        if src.endswith(".hip"):
            cmd += ["-x", "hip", src]
        else:
            cmd += [*CXX_FLAGS, "-x", "c++", src]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
    if verbose and res.stderr.strip():
        print(res.stderr, file=sys.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile LIB from every library source and PROBE_LIB from the probes (always recompiles).
    Returns the library path."""
    _link(SOURCES, LIB, verbose)
    _link(PROBE_SOURCES, PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
