"""The KV migration driven from a plain C99 program, tests/c/gpu_consumer.c.

The program allocates every pool, staging buffer and the workspace with
hipMalloc, creates its own HIP stream, and runs every old rank's pack and
every new rank's unpack through include/remp_kv.h in two layer windows, the
calls after the first reusing the block descriptors.  No Python or torch runs
in that process.  This test writes its inputs (seeded tables and pools),
compiles and runs it, and compares every byte of every new pool and staging
buffer it returns with the oracle.  The program then runs the allocation-free
unpack (remp_kv_unpack_noalloc) of every new rank over the whole cache into
fresh copies of the new pools and checks them byte for byte against what
remp_kv_unpack wrote.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import synthkv
import hostpools
import paper_2606_18741_amd as rk

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
T = oracle.Topology


def _workload(**kw):
    base = dict(name="c_consumer", num_layers=4, num_kv_heads=8, head_dim=64, elem_bytes=2, dtype="u16",
                old_block_size=16, new_block_size=16, num_seqs=6, length_law=("uniform", 0, 200),
                pool_law=("slack", 1.3), old_topo=(2, 1), new_topo=(1, 2), role="all", seed=61)
    base.update(kw)
    return synthkv.KVWorkload(**base)


CASES = {
    "tiny": synthkv.TINY,
    "gqa_tp8_to_tp4pp2_reblock": _workload(head_dim=128, old_topo=(8, 1), new_topo=(4, 2), new_block_size=32),
    "replicated_tp8_to_tp2": _workload(num_kv_heads=4, head_dim=128, old_topo=(8, 1), new_topo=(2, 1)),
}


def _build(tmp_path):
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    lib_dir = os.path.dirname(rk._lib._LIB_PATH)
    exe = tmp_path / "gpu_consumer"
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(rocm, "include"), os.path.join(ROOT, "tests", "c", "gpu_consumer.c"), "-o", str(exe),
           "-L", lib_dir, "-lremp_kv", "-L", os.path.join(rocm, "lib"), "-lamdhip64", f"-Wl,-rpath,{lib_dir}",
           f"-Wl,-rpath,{os.path.join(rocm, 'lib')}"]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    return exe


def _write_inputs(d, w, inp, old_host, new_host):
    ot, nt = inp.old_tables, inp.new_tables
    meta = [w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes, ot.block_size, nt.block_size,
            w.old_topo[0], w.old_topo[1], w.new_topo[0], w.new_topo[1], ot.num_seqs, ot.num_blocks, nt.num_blocks,
            len(ot.ids), len(nt.ids)]
    (d / "meta.txt").write_text(" ".join(str(int(x)) for x in meta) + "\n")
    tables = np.concatenate([ot.seq_lens, ot.offsets, ot.ids, nt.offsets, nt.ids]).astype("<i4")
    tables.tofile(d / "tables.i32")
    for r, layers in old_host.items():
        for l, a in layers.items():
            np.ascontiguousarray(a).tofile(d / f"old_{r}_{l}.bin")
    for q, layers in new_host.items():
        for l, a in layers.items():
            np.ascontiguousarray(a).tofile(d / f"new_{q}_{l}.bin")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
@pytest.mark.parametrize("name", list(CASES))
def test_c_program_migration_matches_oracle(name, tmp_path):
    w = CASES[name]
    inp = synthkv.make_inputs(w)
    L, H = w.num_layers, w.num_kv_heads
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    _write_inputs(tmp_path, w, inp, old_host, new_host)
    exe = _build(tmp_path)
    print(f"[c consumer] {name}: running {exe.name}", flush=True)
    run = subprocess.run([str(exe), str(tmp_path)], capture_output=True, text=True, timeout=120)
    print(run.stdout, run.stderr, flush=True)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "workspace flag 0" in run.stdout
    noalloc = [ln for ln in run.stdout.splitlines() if ln.startswith("no-alloc unpack equal")]
    assert noalloc and int(noalloc[0].split(" on ")[1].split()[0]) > 0, run.stdout

    plan = rk.Plan(w.old_topo, w.new_topo, (L, H, w.head_dim, w.elem_bytes, w.old_block_size, w.new_block_size),
                   rk.HostTables.of(inp.old_tables))
    pairs = [(p.src, p.dst) for p in plan.pairs]
    want_new = hostpools.copy_pools(new_host)
    st = oracle.reshard(old_host, want_new, T(*w.old_topo), T(*w.new_topo), L, H, inp.old_tables, inp.new_tables,
                        pairs=pairs)
    nd = synthkv.numpy_dtype_for(w.elem_bytes)
    for p in pairs:
        want = oracle.staging_buffer(st[p])
        path = tmp_path / f"out_st_{p[0]}_{p[1]}.bin"
        if want.size == 0:
            assert not path.exists()
            continue
        got = np.fromfile(path, dtype=np.uint8)
        assert got.shape == want.shape and np.array_equal(got, want), f"staging {p}"
    for q, layers in want_new.items():
        for l, a in layers.items():
            got = np.fromfile(tmp_path / f"out_new_{q}_{l}.bin", dtype=nd).reshape(a.shape)
            assert np.array_equal(got, a), f"new rank {q} layer {l}"
