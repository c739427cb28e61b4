"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

Every library source is compiled with the host side instrumented (the HIP
sources through hipcc with the sanitizer flags for the host pass only; device
code is built as usual and never runs here), linked with two plain C drivers,
and run:

* tests/c/host_validation.c: planning over many table shapes (padded rows,
  empty sequences, replication, uneven partitions, refused tables) and every
  pack / unpack / local-copy / allocation-free-unpack refusal, plus calls over
  empty layer windows that run the complete host validation of the new tables
  and the slice collection without launching anything;
* tests/c/abi_consumer.c: the host-only ABI walk-through.

Any heap overflow, use after free, leak or undefined behaviour aborts the run.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_18741_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
CLANGXX = os.path.join(ROCM, "llvm", "bin", "clang++")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]
# for hipcc, each host-only flag goes after -Xarch_host so the device pass is built without it
SAN_HOST_ONLY = [x for f in SAN[:3] for x in ("-Xarch_host", f)] + ["-g", "-O1"]
INC = ["-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", os.path.join(ROCM, "include")]


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout + r.stderr


@pytest.mark.skipif(not all(os.path.exists(p) for p in (CLANG, CLANGXX, HIPCC)), reason="ROCm toolchain not found")
def test_host_code_under_asan_and_ubsan(tmp_path):
    d = str(tmp_path)
    objs = []
    for src in ("plan.cpp", "weights_plan.cpp"):
        o = os.path.join(d, src + ".o")
        _run([CLANGXX, *SAN, "-std=c++17", *INC, "-c", os.path.join(CSRC, src), "-o", o], d)
        objs.append(o)
    for src in ("migrate.hip", "weights.hip"):
        o = os.path.join(d, src + ".o")
        _run([HIPCC, "--offload-arch=gfx950", "-std=c++17", *SAN_HOST_ONLY,
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *INC, "-x", "hip",
              os.path.join(CSRC, src), "-c", "-o", o], d)
        objs.append(o)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    for driver, min_ok in (("host_validation.c", 40), ("abi_consumer.c", 15)):
        o = os.path.join(d, driver + ".o")
        exe = os.path.join(d, driver[:-2])
        _run([CLANG, *SAN, "-std=c99", "-Wall", "-Werror", *INC, "-c", os.path.join(ROOT, "tests", "c", driver),
              "-o", o], d)
        _run([CLANGXX, *SAN, o, *objs, "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
              f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe], d)
        r = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
        assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-6000:]
        assert "FAIL" not in r.stdout and r.stdout.count("ok ") >= min_ok, r.stdout
        assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-6000:]
