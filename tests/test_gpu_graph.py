"""The KV entry points under HIP graph capture.

pack, unpack and copy_local enqueue kernels only (no allocation, no memset,
no synchronisation), so a whole migration step can be captured once and
replayed.  Each replay must reproduce the oracle's result; between replays
the destination pools and staging are overwritten eagerly, so a replay that
skipped or reused work would show.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synthkv
import hostpools
from gpu_harness import (DeviceTables, RankPool, Workspace, log, rank_layers, shape_of, staging_for_pairs,
                         window_args)

pytestmark = pytest.mark.gpu
T = oracle.Topology


def _rk():
    import paper_2606_18741_amd as rk
    return rk


def _setup(w):
    rk = _rk()
    inp = synthkv.make_inputs(w)
    L = w.num_layers
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    src = {r: RankPool.from_host(old_host[r], rank_layers(r, w.old_topo, L), inp.old_tables.num_blocks, r)
           for r in range(plan.info.old_world)}
    dst = {q: RankPool.from_host(new_host[q], rank_layers(q, w.new_topo, L), inp.new_tables.num_blocks, q)
           for q in range(plan.info.new_world)}
    return inp, plan, dto, dtn, src, dst, old_host, new_host


def _check(w, inp, plan, dst, old_host, new_host):
    want = hostpools.copy_pools(new_host)
    oracle.reshard(old_host, want, T(*w.old_topo), T(*w.new_topo), w.num_layers, w.num_kv_heads,
                   inp.old_tables, inp.new_tables)
    for q, pool in dst.items():
        got = pool.host(w.elem_bytes)
        for l, a in want[q].items():
            assert np.array_equal(got[l], a), f"new rank {q} layer {l}"


def _reset(dst, new_host, staging):
    for q, pool in dst.items():
        for l, t in pool.store.items():
            t.copy_(torch.from_numpy(new_host[q][l].view(t.cpu().numpy().dtype)))
    for b in staging.values():
        b.fill_(0x5A)


@pytest.mark.parametrize("local", [False, True])
@pytest.mark.parametrize("name,windows", [("tiny", None), ("gqa70b", 8), ("mha7b", 4)])
def test_graph_replays_match_oracle(name, windows, local):
    _graph_case(name, windows, local, reuse=False)


@pytest.mark.parametrize("local", [False, True])
@pytest.mark.parametrize("name,windows", [("gqa70b", 8), ("mha7b", 4)])
def test_graph_replays_with_descriptor_reuse(name, windows, local):
    """Only the first pack and unpack of the captured step expand the tables; the workspace is cleared
    between replays, so every replay must write the descriptors and their stamps again."""
    _graph_case(name, windows, local, reuse=True)


def _graph_case(name, windows, local, reuse):
    rk = _rk()
    w = synthkv.WORKLOADS[name]
    if name != "tiny":
        w = synthkv.reduced(w, num_seqs=4, max_len=200)
    L = w.num_layers
    inp, plan, dto, dtn, src, dst, old_host, new_host = _setup(w)
    W_old, W_new = plan.info.old_world, plan.info.new_world
    pairs = [(p.src, p.dst) for p in plan.pairs if not (local and p.src == p.dst)]
    staging = staging_for_pairs(plan, w.seed, pairs)
    ws = Workspace(plan)
    step = L // windows if windows else L
    wins = [(a, min(L, a + step)) for a in range(0, L, step)]
    fl = rk.REMP_KV_SKIP_LOCAL if local else 0
    ru = rk.REMP_KV_REUSE_DESCRIPTORS if reuse else 0
    args = [(l0, l1, {r: window_args(plan, staging, r, W_new, True, l0, l1) for r in range(W_old)},
             {q: window_args(plan, staging, q, W_old, False, l0, l1) for q in range(W_new)}) for (l0, l1) in wins]

    def migrate(stream):
        for i, (l0, l1, outs, ins) in enumerate(args):
            for r in range(W_old):
                again = ru if (i or r) else 0
                plan.pack(r, src[r].arg, dto.dev, outs[r], ws.buf, ws.bytes, stream, l0, l1, flags=fl | again)
            for q in range(W_new):
                again = ru if (i or q) else 0
                plan.unpack(q, ins[q], dst[q].arg, dtn.host, dtn.dev, ws.buf, ws.bytes, stream, l0, l1,
                            flags=fl | again)
            if local:
                for r in range(min(W_old, W_new)):
                    plan.copy_local(r, src[r].arg, dto.dev, dst[r].arg, dtn.host, dtn.dev, ws.buf, ws.bytes, stream,
                                    l0, l1, flags=ru)

    log(f"[graph] capture {w.name} windows={len(wins)} local={local} reuse={reuse}")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):          # warm-up outside the capture
        migrate(side.cuda_stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        migrate(side.cuda_stream)
    torch.cuda.synchronize()
    for rep in range(3):
        _reset(dst, new_host, staging)
        if reuse:
            ws.buf.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert ws.flag() == 0
        _check(w, inp, plan, dst, old_host, new_host)
        log(f"[graph] replay {rep} matches the oracle")
