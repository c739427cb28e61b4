"""The C ABI from a plain C99 program (no Python, no torch): tests/c/abi_consumer.c is compiled
with gcc against include/*.h and linked with the built library, then run (host-only calls)."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

import paper_2606_18741_amd as rk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c99_consumer(tmp_path):
    lib_dir = os.path.dirname(rk._lib._LIB_PATH)
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    exe = tmp_path / "abi_consumer"
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(rocm, "include"), os.path.join(ROOT, "tests", "c", "abi_consumer.c"), "-o", str(exe),
           "-L", lib_dir, "-lremp_kv", f"-Wl,-rpath,{lib_dir}"]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "FAIL" not in run.stdout and run.stdout.count("ok ") >= 15, run.stdout
    # every constant of the headers has the same value in the Python binding
    consts = {ln.split()[1]: int(ln.split()[2]) for ln in run.stdout.splitlines() if ln.startswith("const ")}
    assert len(consts) == 19, consts
    status_by_name = {v: k for k, v in rk._lib.STATUS.items()}
    for name, value in consts.items():
        if name.startswith("REMP_E_") or name == "REMP_OK":
            assert status_by_name[name] == value, name
        else:
            py = name.replace("REMP_KV_LAYOUT_", "LAYOUT_")
            assert getattr(rk._lib, py) == value, name
