"""GPU parity: libremp_kv.so's pack and unpack against the CPU oracle, bit for bit.

Small and reduced workloads run every old rank's pack and every new rank's
unpack on the one GPU and compare every staging byte and every byte of every
new pool (live slots and untouched sentinels alike) with the oracle; the
source pools must come back unchanged.  Two hand-derived examples are also
checked against their hand-written expected values directly.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

import oracle
import synthkv
from synthkv import tables_from_rows

import hostpools
from gpu_harness import (DeviceTables, RankPool, Workspace, log, rank_layers, shape_of, stream_handle,
                         staging_for_pairs, window_args)

pytestmark = pytest.mark.gpu

from edgecases import EDGE, SHIFTED_LAYOUTS, custom as _custom, shifted_old_lengths_case

T = oracle.Topology
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rk():
    import paper_2606_18741_amd as rk
    return rk


def migrate_all(w, old_tables, new_tables, old_host, new_host, windows=None, local=False, reuse=False):
    """Pack every old rank, unpack every new rank, per layer window.  Returns device state.

    local: pack and unpack skip the slices a rank keeps, and remp_kv_copy_local
    moves those pool to pool.
    reuse: only the first pack and the first unpack expand the block tables;
    every later call (and every local copy) reuses their descriptors.
    """
    rk = _rk()
    L = w.num_layers
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(old_tables))
    dto, dtn = DeviceTables(old_tables), DeviceTables(new_tables)
    W_old, W_new = plan.info.old_world, plan.info.new_world
    src = {r: RankPool.from_host(old_host[r], rank_layers(r, w.old_topo, L), old_tables.num_blocks, r)
           for r in range(W_old)}
    dst = {q: RankPool.from_host(new_host[q], rank_layers(q, w.new_topo, L), new_tables.num_blocks, q)
           for q in range(W_new)}
    pairs = [(p.src, p.dst) for p in plan.pairs if not (local and p.src == p.dst)]
    staging = staging_for_pairs(plan, w.seed, pairs)
    ws = Workspace(plan)
    stream = stream_handle()
    flags = []
    fl = rk.REMP_KV_SKIP_LOCAL if local else 0
    reuse_fl = rk.REMP_KV_REUSE_DESCRIPTORS if reuse else 0
    first_pack = first_unpack = True
    for (l0, l1) in (windows or [(0, L)]):
        for r in range(W_old):
            plan.pack(r, src[r].arg, dto.dev, window_args(plan, staging, r, W_new, True, l0, l1),
                      ws.buf, ws.bytes, stream, l0, l1, flags=fl | (0 if first_pack else reuse_fl))
            first_pack = first_pack and l0 == l1
        torch.cuda.synchronize()
        flags.append(ws.flag())
        for q in range(W_new):
            plan.unpack(q, window_args(plan, staging, q, W_old, False, l0, l1), dst[q].arg, dtn.host, dtn.dev,
                        ws.buf, ws.bytes, stream, l0, l1, flags=fl | (0 if first_unpack else reuse_fl))
            first_unpack = first_unpack and l0 == l1
        torch.cuda.synchronize()
        flags.append(ws.flag())
        if local:
            for r in range(min(W_old, W_new)):
                plan.copy_local(r, src[r].arg, dto.dev, dst[r].arg, dtn.host, dtn.dev, ws.buf, ws.bytes, stream,
                                l0, l1, flags=reuse_fl)
            torch.cuda.synchronize()
            flags.append(ws.flag())
    return plan, src, dst, staging, flags


def check_against_oracle(w, inp, windows=None, log_name="", local=False, identical_replicas=True, reuse=False):
    L, H = w.num_layers, w.num_kv_heads
    old_host = hostpools.source_pools(w, inp.old_tables, identical_replicas=identical_replicas)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    log(f"[parity] {log_name or w.name}: T={int(inp.lens.sum())} windows={windows} local={local} reuse={reuse}")
    plan, src, dst, staging, flags = migrate_all(w, inp.old_tables, inp.new_tables, old_host, new_host, windows,
                                                 local, reuse)
    pairs = [(p.src, p.dst) for p in plan.pairs if not (local and p.src == p.dst)]
    st = oracle.reshard(old_host, new_host, T(*w.old_topo), T(*w.new_topo), L, H, inp.old_tables,
                        inp.new_tables, pairs=pairs)
    assert all(f == 0 for f in flags), flags
    for p in pairs:
        want = oracle.staging_buffer(st[p])
        if want.size == 0:
            assert p not in staging or staging[p].numel() == 0
            continue
        got = staging[p].cpu().numpy()
        assert got.shape == want.shape, (p, got.shape, want.shape)
        if not np.array_equal(got, want):
            bad = np.nonzero(got != want)[0]
            pytest.fail(f"staging {p}: {bad.size} bytes differ, first at {bad[0]}")
    for q, pool in dst.items():
        got = pool.host(w.elem_bytes)
        for l, a in new_host[q].items():
            if not np.array_equal(got[l], a):
                bad = np.argwhere(got[l] != a)
                pytest.fail(f"new rank {q} layer {l}: {len(bad)} elements differ, first at {bad[0].tolist()}")
    for r, pool in src.items():           # pack never writes its source
        got = pool.host(w.elem_bytes)
        for l, a in old_host[r].items():
            assert np.array_equal(got[l], a), f"source rank {r} layer {l} modified"


# ---------------------------------------------------------------------------
# hand-derived examples (expected values written by hand, not by the oracle)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["hand_tp2pp1_to_tp1pp2.json", "hand_tp1pp2_to_tp2pp1_reblock.json",
                                  "hand_replicated_tp4_to_tp2.json"])
def test_golden_hand_example_gpu(name):
    with open(os.path.join(GOLDEN, name)) as f:
        g = json.load(f)
    w = synthkv.KVWorkload(name="golden", num_layers=g["num_layers"], num_kv_heads=g["num_kv_heads"],
                           head_dim=g["head_dim"], elem_bytes=2, dtype="u16", old_block_size=g["old_block_size"],
                           new_block_size=g["new_block_size"], num_seqs=len(g["seq_lens"]),
                           length_law=("fixed", 0), pool_law=("fixed", 0), old_topo=tuple(g["old_topo"]),
                           new_topo=tuple(g["new_topo"]), role="all", seed=0)
    old_t = tables_from_rows(g["seq_lens"], g["old_rows"], g["old_num_blocks"], g["old_block_size"])
    new_t = tables_from_rows(g["seq_lens"], g["new_rows"], g["new_num_blocks"], g["new_block_size"])
    old_host = {}
    for key, arr in g["old_pools"].items():
        r, l = map(int, key.split(":"))
        old_host.setdefault(r, {})[l] = np.array(arr, dtype=np.uint16)
    new_host = {}
    nt = T(*g["new_topo"])
    for q in range(nt.world):
        for l in rank_layers(q, g["new_topo"], g["num_layers"]):
            new_host.setdefault(q, {})[l] = np.full(
                (2, g["new_num_blocks"], g["new_block_size"], len(oracle.heads_of(q, nt, g["num_kv_heads"])),
                 g["head_dim"]), g["sentinel"], np.uint16)
    log(f"[golden] {name}")
    plan, src, dst, staging, flags = migrate_all(w, old_t, new_t, old_host, new_host)
    assert all(f == 0 for f in flags)
    for key, arr in g["expected_new_pools"].items():
        q, l = map(int, key.split(":"))
        np.testing.assert_array_equal(dst[q].host(2)[l], np.array(arr, dtype=np.uint16), err_msg=key)
    for key, vals in g["expected_staging"].items():
        r, q = map(int, key.split(":"))
        np.testing.assert_array_equal(staging[(r, q)].cpu().numpy().view(np.uint16),
                                      np.array(vals, dtype=np.uint16), err_msg=key)


# ---------------------------------------------------------------------------
# the five workloads (Tiny at full size; the others with a small population)
# ---------------------------------------------------------------------------

def test_tiny_all_ranks():
    w = synthkv.TINY
    check_against_oracle(w, synthkv.make_inputs(w))


@pytest.mark.parametrize("name", ["mha7b", "mha13b", "gqa70b", "gqa70b_long", "qwen30b", "ds32b"])
def test_reduced_workload_all_ranks(name):
    w = synthkv.reduced(synthkv.WORKLOADS[name], num_seqs=5, max_len=300)
    check_against_oracle(w, synthkv.make_inputs(w))


def test_layer_windows_match_whole():
    w = synthkv.reduced(synthkv.GQA_70B_LONG, num_seqs=3, max_len=200)
    check_against_oracle(w, synthkv.make_inputs(w), windows=[(0, 1), (1, 7), (7, 40), (40, 41), (41, 80)])


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(EDGE))
def test_edge_case(name):
    w = EDGE[name]
    check_against_oracle(w, synthkv.make_inputs(w), log_name=name)


@pytest.mark.parametrize("name", [n for n in EDGE if n.startswith("replicated")])
def test_replica_choice_visible(name):
    """Replicas hold different bytes, so the source replica each new rank used is checked too."""
    check_against_oracle(EDGE[name], synthkv.make_inputs(EDGE[name]), log_name=name + "_distinct",
                         identical_replicas=False)


@pytest.mark.parametrize("name", ["replicated_tp8_to_tp2", "replicated_keep_local"])
def test_replica_choice_visible_local(name):
    check_against_oracle(EDGE[name], synthkv.make_inputs(EDGE[name]), log_name=name + "_distinct_local",
                         identical_replicas=False, local=True)


def test_padded_table_rows():
    w = _custom(num_seqs=7)
    check_against_oracle(w, synthkv.make_inputs(w, row_pad=3), log_name="padded_rows")


def test_unpack_from_oracle_staging():
    """Unpack alone, fed staging the oracle wrote (independent of the pack kernel)."""
    rk = _rk()
    w = synthkv.reduced(synthkv.GQA_70B, num_seqs=4, max_len=150)
    inp = synthkv.make_inputs(w)
    L, H = w.num_layers, w.num_kv_heads
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    pre = hostpools.copy_pools(new_host)
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    pairs = [(p.src, p.dst) for p in plan.pairs]
    st = oracle.reshard(old_host, new_host, T(*w.old_topo), T(*w.new_topo), L, H, inp.old_tables,
                        inp.new_tables, pairs=pairs)
    staging = {p: torch.from_numpy(oracle.staging_buffer(st[p]).copy()).cuda() for p in pairs}
    dtn = DeviceTables(inp.new_tables)
    ws = Workspace(plan)
    for q in range(plan.info.new_world):
        dst = RankPool.from_host(pre[q], rank_layers(q, w.new_topo, L), inp.new_tables.num_blocks, q)
        plan.unpack(q, window_args(plan, staging, q, plan.info.old_world, False, 0, L), dst.arg, dtn.host,
                    dtn.dev, ws.buf, ws.bytes, stream_handle())
        torch.cuda.synchronize()
        assert ws.flag() == 0
        got = dst.host(2)
        for l in new_host[q]:
            np.testing.assert_array_equal(got[l], new_host[q][l])


def test_mismatched_device_tables_are_contained():
    """Device tables that disagree with the host ones must not fault; the flag reports it."""
    rk = _rk()
    w = synthkv.reduced(synthkv.TINY, num_seqs=3, max_len=60)
    inp = synthkv.make_inputs(w)
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    old_host = hostpools.source_pools(w, inp.old_tables)
    src = RankPool.from_host(old_host[0], rank_layers(0, w.old_topo, w.num_layers), inp.old_tables.num_blocks, 0)
    dto = DeviceTables(inp.old_tables)
    dto.ids.fill_(1 << 30)                 # every id out of range on the device only
    pairs = [(p.src, p.dst) for p in plan.pairs]
    staging = staging_for_pairs(plan, w.seed, pairs)
    before = {p: b.clone() for p, b in staging.items()}
    ws = Workspace(plan)
    plan.pack(0, src.arg, dto.dev, window_args(plan, staging, 0, plan.info.new_world, True, 0, w.num_layers),
              ws.buf, ws.bytes, stream_handle())
    torch.cuda.synchronize()
    assert ws.flag() != 0
    for p in pairs:                        # nothing was copied
        assert torch.equal(staging[p], before[p])


@pytest.mark.parametrize("lo,ln,bn", SHIFTED_LAYOUTS)
def test_local_copy_contains_shifted_device_lengths(lo, ln, bn):
    """Old device lengths that shift a sequence start (same total) give some rows of the local copies a
    negative token index; those rows must be skipped and flagged, never read from before an old block.
    (The CPU model of the kernels checks this case access by access: test_model_shifted_old_lengths.)"""
    rk = _rk()
    w, inp, (lens, offs, ids) = shifted_old_lengths_case(bn)
    L = w.num_layers
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    dto = DeviceTables(inp.old_tables)
    dto.lens.copy_(torch.from_numpy(lens))
    dto.ids.copy_(torch.from_numpy(ids))
    dtn = DeviceTables(inp.new_tables)
    ws = Workspace(plan)
    W = plan.info.old_world
    src = {r: _upload_layout(old_host[r], lo, rank_layers(r, w.old_topo, L), inp.old_tables.num_blocks)
           for r in range(W)}
    dst = {q: _upload_layout(new_host[q], ln, rank_layers(q, w.new_topo, L), inp.new_tables.num_blocks)
           for q in range(W)}
    flags = []
    for r in range(W):
        plan.copy_local(r, src[r][0], dto.dev, dst[r][0], dtn.host, dtn.dev, ws.buf, ws.bytes, stream_handle())
        torch.cuda.synchronize()
        flags.append(ws.flag())
    assert all(f == 1 for f in flags), flags
    nd = synthkv.numpy_dtype_for(w.elem_bytes)
    for r in range(W):                    # sources untouched
        for l, (kt, vt) in src[r][1].items():
            want = oracle.encode_pool(old_host[r][l], lo)
            assert np.array_equal(kt.cpu().numpy().view(nd), want[0])
            assert np.array_equal(vt.cpu().numpy().view(nd), want[1])
    live = np.zeros((inp.new_tables.num_blocks, inp.new_tables.block_size), bool)
    for s_ in range(len(inp.lens)):
        blk, slot = oracle.token_slots(inp.new_tables, s_)
        live[blk, slot] = True
    for q in range(W):                    # dead slots of the new pools untouched
        for l, (kt, vt) in dst[q][1].items():
            got = oracle.decode_pool([kt.cpu().numpy().view(nd), vt.cpu().numpy().view(nd)], ln)
            assert np.array_equal(got[:, ~live], new_host[q][l][:, ~live]), f"rank {q} layer {l}: a dead slot written"


# ---------------------------------------------------------------------------
# local fast path: slices a rank keeps move pool to pool, the rest through staging
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny", "mha7b", "mha13b", "gqa70b", "gqa70b_long", "qwen30b", "ds32b"])
def test_local_fast_path(name):
    w = synthkv.WORKLOADS[name]
    if name != "tiny":
        w = synthkv.reduced(w, num_seqs=5, max_len=300)
    check_against_oracle(w, synthkv.make_inputs(w), local=True)


@pytest.mark.parametrize("name", list(EDGE))
def test_local_fast_path_edge_case(name):
    check_against_oracle(EDGE[name], synthkv.make_inputs(EDGE[name]), log_name=name, local=True)


def test_local_fast_path_windows():
    w = synthkv.reduced(synthkv.GQA_70B, num_seqs=3, max_len=200)
    check_against_oracle(w, synthkv.make_inputs(w), windows=[(0, 13), (13, 40), (40, 80)], local=True)


@pytest.mark.parametrize("wg_bytes", [2048, 8192, 32768, 262144, 1 << 20])
@pytest.mark.parametrize("name", ["mha7b", "gqa70b", "merged_rows_mha"])
def test_workgroup_sizes(name, wg_bytes, monkeypatch):
    """Bit-exact at other bytes-per-workgroup targets (REMP_KV_WG_BYTES, a tuning override): one to
    many units per workgroup and ragged last workgroups, for the small-unit (GQA) and large-unit (MHA)
    launch shapes, staged and with the local fast path."""
    w = EDGE[name] if name in EDGE else synthkv.reduced(synthkv.WORKLOADS[name], num_seqs=4, max_len=250)
    monkeypatch.setenv("REMP_KV_WG_BYTES", str(wg_bytes))
    inp = synthkv.make_inputs(w)
    check_against_oracle(w, inp, log_name=f"{name} wg {wg_bytes}")
    check_against_oracle(w, inp, log_name=f"{name} wg {wg_bytes} local", local=True)


# ---------------------------------------------------------------------------
# pool layouts: HND and the ROCm paged-attention layout go through LDS tiles
# ---------------------------------------------------------------------------

def _upload_layout(arrays, layout, layers_of_rank, num_blocks):
    """Encode host [2, nb, bs, H, D] arrays into `layout` and upload K and V separately."""
    rk = _rk()
    ks, vs, keep = [], [], {}
    for l in layers_of_rank:
        if l not in arrays:
            ks.append(None)
            vs.append(None)
            continue
        k, v = oracle.encode_pool(arrays[l], layout)
        signed = {1: np.int8, 2: np.int16, 4: np.int32}[k.dtype.itemsize]
        kt = torch.from_numpy(np.ascontiguousarray(k).view(signed)).cuda()
        vt = torch.from_numpy(np.ascontiguousarray(v).view(signed)).cuda()
        keep[l] = (kt, vt)
        ks.append(kt)
        vs.append(vt)
    return rk.PoolArg(ks, vs, num_blocks, layout=layout), keep


LAYOUT_CASES = [(0, 1), (1, 0), (0, 2), (2, 0), (2, 2), (1, 2), (2, 1)]


def _layout_workload(shape):
    base = dict(name="layout", num_layers=4, num_kv_heads=8, head_dim=128, elem_bytes=2, dtype="bf16",
                old_block_size=16, new_block_size=16, num_seqs=5, length_law=("uniform", 0, 150),
                pool_law=("slack", 1.3), old_topo=(8, 1), new_topo=(4, 2), role="all", seed=41)
    extra = {"gqa70b": {}, "mha7b_reblock": dict(num_kv_heads=16, old_topo=(4, 1), new_topo=(2, 2),
                                                 new_block_size=32),
             "fp8": dict(elem_bytes=1, dtype="fp8", old_block_size=16, new_block_size=32),
             "replicated": dict(num_kv_heads=4, old_topo=(8, 1), new_topo=(2, 2)),
             "shrink": dict(num_kv_heads=4, old_topo=(4, 1), new_topo=(2, 1), old_block_size=32,
                            new_block_size=16)}[shape]
    base.update(extra)
    return synthkv.KVWorkload(**base)


@pytest.mark.parametrize("lo,ln", LAYOUT_CASES)
@pytest.mark.parametrize("shape", ["gqa70b", "mha7b_reblock", "fp8", "replicated"])
def test_layouts(shape, lo, ln):
    _layouts_case(shape, lo, ln, reuse=False)


@pytest.mark.parametrize("lo,ln", [(1, 2), (2, 1)])
@pytest.mark.parametrize("shape", ["gqa70b", "mha7b_reblock"])
def test_layouts_reuse(shape, lo, ln):
    """Head-tile copies with descriptors reused after the first pack and the first unpack."""
    _layouts_case(shape, lo, ln, reuse=True)


def _layouts_case(shape, lo, ln, reuse):
    """shape: a name of _layout_workload, or a workload."""
    rk = _rk()
    w = shape if isinstance(shape, synthkv.KVWorkload) else _layout_workload(shape)
    shape = shape if isinstance(shape, str) else w.name
    inp = synthkv.make_inputs(w)
    L, H = w.num_layers, w.num_kv_heads
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    log(f"[layout] {shape} old {lo} new {ln} reuse {reuse}")
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    W_old, W_new = plan.info.old_world, plan.info.new_world
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    src = {r: _upload_layout(old_host[r], lo, rank_layers(r, w.old_topo, L), inp.old_tables.num_blocks)
           for r in range(W_old)}
    dst = {q: _upload_layout(new_host[q], ln, rank_layers(q, w.new_topo, L), inp.new_tables.num_blocks)
           for q in range(W_new)}
    pairs = [(p.src, p.dst) for p in plan.pairs]
    staging = staging_for_pairs(plan, w.seed, pairs)
    ws = Workspace(plan)
    ru = rk.REMP_KV_REUSE_DESCRIPTORS if reuse else 0
    for r in range(W_old):
        plan.pack(r, src[r][0], dto.dev, window_args(plan, staging, r, W_new, True, 0, L), ws.buf, ws.bytes,
                  stream_handle(), flags=ru if r else 0)
    for q in range(W_new):
        plan.unpack(q, window_args(plan, staging, q, W_old, False, 0, L), dst[q][0], dtn.host, dtn.dev, ws.buf,
                    ws.bytes, stream_handle(), flags=ru if q else 0)
    torch.cuda.synchronize()
    assert ws.flag() == 0
    st = oracle.reshard(old_host, new_host, T(*w.old_topo), T(*w.new_topo), L, H, inp.old_tables,
                        inp.new_tables, pairs=pairs)
    for p in pairs:
        want = oracle.staging_buffer(st[p])
        if want.size:
            assert np.array_equal(staging[p].cpu().numpy(), want), f"staging {p}"
    nd = synthkv.numpy_dtype_for(w.elem_bytes)
    for q in range(W_new):
        for l, (kt, vt) in dst[q][1].items():
            want = oracle.encode_pool(new_host[q][l], ln)
            assert np.array_equal(kt.cpu().numpy().view(nd), want[0]), f"new rank {q} layer {l} K"
            assert np.array_equal(vt.cpu().numpy().view(nd), want[1]), f"new rank {q} layer {l} V"
    for r in range(W_old):                # sources untouched
        for l, (kt, vt) in src[r][1].items():
            want = oracle.encode_pool(old_host[r][l], lo)
            assert np.array_equal(kt.cpu().numpy().view(nd), want[0])
            assert np.array_equal(vt.cpu().numpy().view(nd), want[1])


@pytest.mark.parametrize("lo,ln", LAYOUT_CASES + [(1, 1)])
@pytest.mark.parametrize("shape", ["gqa70b", "mha7b_reblock", "fp8", "replicated", "shrink"])
def test_local_fast_path_layouts(shape, lo, ln):
    """Local fast path with HND / ROCm pools: pack and unpack skip the local slices, copy_local moves them
    through head tiles; every byte of every new pool must equal the oracle's, in the new layout."""
    _local_layouts_case(shape, lo, ln, reuse=False)


@pytest.mark.parametrize("lo,ln", [(1, 2), (2, 1), (1, 1)])
@pytest.mark.parametrize("shape", ["gqa70b", "replicated"])
def test_local_fast_path_layouts_reuse(shape, lo, ln):
    """The same with the block descriptors reused by every call after the first pack and unpack."""
    _local_layouts_case(shape, lo, ln, reuse=True)


def _local_layouts_case(shape, lo, ln, reuse):
    """shape: a name of _layout_workload, or a workload."""
    rk = _rk()
    w = shape if isinstance(shape, synthkv.KVWorkload) else _layout_workload(shape)
    shape = shape if isinstance(shape, str) else w.name
    inp = synthkv.make_inputs(w)
    L, H = w.num_layers, w.num_kv_heads
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    log(f"[local layout] {shape} old {lo} new {ln} reuse {reuse}")
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    W_old, W_new = plan.info.old_world, plan.info.new_world
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    src = {r: _upload_layout(old_host[r], lo, rank_layers(r, w.old_topo, L), inp.old_tables.num_blocks)
           for r in range(W_old)}
    dst = {q: _upload_layout(new_host[q], ln, rank_layers(q, w.new_topo, L), inp.new_tables.num_blocks)
           for q in range(W_new)}
    pairs = [(p.src, p.dst) for p in plan.pairs if p.src != p.dst]
    staging = staging_for_pairs(plan, w.seed, pairs)
    ws = Workspace(plan)
    fl = rk.REMP_KV_SKIP_LOCAL
    ru = rk.REMP_KV_REUSE_DESCRIPTORS if reuse else 0
    for r in range(W_old):
        plan.pack(r, src[r][0], dto.dev, window_args(plan, staging, r, W_new, True, 0, L), ws.buf, ws.bytes,
                  stream_handle(), flags=fl | (ru if r else 0))
    torch.cuda.synchronize()
    assert ws.flag() == 0
    for q in range(W_new):
        plan.unpack(q, window_args(plan, staging, q, W_old, False, 0, L), dst[q][0], dtn.host, dtn.dev, ws.buf,
                    ws.bytes, stream_handle(), flags=fl | (ru if q else 0))
    torch.cuda.synchronize()
    assert ws.flag() == 0
    for r in range(min(W_old, W_new)):
        plan.copy_local(r, src[r][0], dto.dev, dst[r][0], dtn.host, dtn.dev, ws.buf, ws.bytes, stream_handle(),
                        flags=ru)
    torch.cuda.synchronize()
    assert ws.flag() == 0
    oracle.reshard(old_host, new_host, T(*w.old_topo), T(*w.new_topo), L, H, inp.old_tables, inp.new_tables)
    nd = synthkv.numpy_dtype_for(w.elem_bytes)
    for q in range(W_new):
        for l, (kt, vt) in dst[q][1].items():
            want = oracle.encode_pool(new_host[q][l], ln)
            assert np.array_equal(kt.cpu().numpy().view(nd), want[0]), f"new rank {q} layer {l} K"
            assert np.array_equal(vt.cpu().numpy().view(nd), want[1]), f"new rank {q} layer {l} V"
    for r in range(W_old):                # sources untouched
        for l, (kt, vt) in src[r][1].items():
            want = oracle.encode_pool(old_host[r][l], lo)
            assert np.array_equal(kt.cpu().numpy().view(nd), want[0])
            assert np.array_equal(vt.cpu().numpy().view(nd), want[1])


# ---------------------------------------------------------------------------
# descriptor reuse across calls (REMP_KV_REUSE_DESCRIPTORS)
# ---------------------------------------------------------------------------

REUSE_CASES = {
    # per-layer windows of a layer merge plus head split (staged)
    "gqa70b_long_layers": (lambda: synthkv.reduced(synthkv.GQA_70B_LONG, num_seqs=3, max_len=200),
                           [(l, l + 1) for l in range(10)] + [(10, 17), (17, 40), (40, 41), (41, 80)], False),
    "gqa70b_windows_local": (lambda: synthkv.reduced(synthkv.GQA_70B, num_seqs=5, max_len=300),
                             [(0, 13), (13, 13), (13, 40), (40, 80)], True),
    "mha7b_rows_windows": (lambda: synthkv.reduced(synthkv.MHA_7B, num_seqs=4, max_len=200),
                           [(0, 5), (5, 16), (16, 32)], False),
    "replicated_local": (lambda: EDGE["replicated_keep_local"], [(0, 3), (3, 8)], True),
    "reblock_local": (lambda: EDGE["heads_not_nested_reblock"], [(0, 2), (2, 6)], True),
    "uneven_pp_local": (lambda: EDGE["uneven_pp"], [(0, 1), (1, 4), (4, 5)], True),
}


def _windows_cover(windows, L):
    cov = sorted((a, b) for a, b in windows if a < b)
    assert cov[0][0] == 0 and cov[-1][1] == L and all(x[1] == y[0] for x, y in zip(cov, cov[1:])), cov


@pytest.mark.parametrize("name", list(REUSE_CASES))
def test_reuse_descriptors_windows(name):
    """Windows where only the first pack and unpack expand the tables give the oracle's bytes."""
    make, windows, local = REUSE_CASES[name]
    w = make()
    _windows_cover(windows, w.num_layers)
    check_against_oracle(w, synthkv.make_inputs(w), windows=windows, local=local, reuse=True, log_name=name)


def _reuse_setup(w, inp):
    rk = _rk()
    L = w.num_layers
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    old_host = hostpools.source_pools(w, inp.old_tables)
    new_host = hostpools.sentinel_pools(w, inp.new_tables)
    src = {r: RankPool.from_host(old_host[r], rank_layers(r, w.old_topo, L), inp.old_tables.num_blocks, r)
           for r in range(plan.info.old_world)}
    dst = {q: RankPool.from_host(new_host[q], rank_layers(q, w.new_topo, L), inp.new_tables.num_blocks, q)
           for q in range(plan.info.new_world)}
    pairs = [(p.src, p.dst) for p in plan.pairs]
    staging = staging_for_pairs(plan, w.seed, pairs)
    return plan, old_host, new_host, src, dst, pairs, staging


def _unchanged(staging, before, dst, new_host, elem_bytes):
    for p in before:
        assert torch.equal(staging[p], before[p]), f"staging {p} written"
    for q, pool in dst.items():
        got = pool.host(elem_bytes)
        for l, a in new_host[q].items():
            assert np.array_equal(got[l], a), f"new rank {q} layer {l} written"


@pytest.mark.parametrize("fill", ["zeros", "random"])
def test_reuse_without_expansion_copies_nothing(fill):
    _reuse_stale_case(fill, layout=0)


def test_reuse_without_expansion_copies_nothing_hnd():
    """The same for head-tile kernels (HND pools)."""
    _reuse_stale_case("random", layout=1)


def _reuse_stale_case(fill, layout):
    """A reusing call on a workspace that holds no matching descriptors copies nothing and sets flag 2."""
    rk = _rk()
    w = synthkv.reduced(synthkv.TINY, num_seqs=4, max_len=120)
    inp = synthkv.make_inputs(w)
    L = w.num_layers
    plan, old_host, new_host, src, dst, pairs, staging = _reuse_setup(w, inp)
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    before = {p: b.clone() for p, b in staging.items()}
    ws = Workspace(plan)
    if fill == "random":
        g = torch.Generator().manual_seed(5)
        ws.buf.copy_(torch.randint(0, 256, (ws.bytes,), generator=g, dtype=torch.uint8))
        ws.set_flag(0)
    else:
        ws.buf.zero_()
    reuse = rk.REMP_KV_REUSE_DESCRIPTORS
    # the same storage read as `layout` (HND selects the head-tile kernels; nothing may be written anyway)
    src_arg = rk.PoolArg(list(src[0].arg._k), list(src[0].arg._v), inp.old_tables.num_blocks, layout=layout)
    dst_arg = rk.PoolArg(list(dst[0].arg._k), list(dst[0].arg._v), inp.new_tables.num_blocks, layout=layout)
    log(f"[reuse] no expansion, workspace {fill}, layout {layout}")
    plan.pack(0, src_arg, dto.dev, window_args(plan, staging, 0, plan.info.new_world, True, 0, L), ws.buf,
              ws.bytes, stream_handle(), flags=reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 2
    ws.set_flag(0)
    plan.unpack(0, window_args(plan, staging, 0, plan.info.old_world, False, 0, L), dst_arg, dtn.host, dtn.dev,
                ws.buf, ws.bytes, stream_handle(), flags=reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 2
    ws.set_flag(0)
    plan.copy_local(0, src_arg, dto.dev, dst_arg, dtn.host, dtn.dev, ws.buf, ws.bytes, stream_handle(),
                    flags=reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 2
    _unchanged(staging, before, dst, new_host, w.elem_bytes)


def test_reuse_refuses_other_tables_and_plans():
    """Descriptors of other new tables, or of another plan, are not reused; the matching ones are."""
    rk = _rk()
    w = synthkv.reduced(synthkv.GQA_70B, num_seqs=4, max_len=150)
    inp = synthkv.make_inputs(w)
    L, H = w.num_layers, w.num_kv_heads
    plan, old_host, new_host, src, dst, pairs, staging = _reuse_setup(w, inp)
    W_old, W_new = plan.info.old_world, plan.info.new_world
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    # other new tables with the same lengths: the same blocks in another order
    rows = [inp.new_tables.row(s) for s in range(inp.new_tables.num_seqs)]
    ids = np.concatenate(rows)[::-1].copy()
    k, rows_b = 0, []
    for r in rows:
        rows_b.append(ids[k:k + len(r)])
        k += len(r)
    tables_b = tables_from_rows(inp.new_tables.seq_lens, rows_b, inp.new_tables.num_blocks,
                                inp.new_tables.block_size)
    dtb = DeviceTables(tables_b)
    ws = Workspace(plan)
    reuse = rk.REMP_KV_REUSE_DESCRIPTORS
    stream = stream_handle()
    for r in range(W_old):                 # the first pack expands; the rest reuse
        plan.pack(r, src[r].arg, dto.dev, window_args(plan, staging, r, W_new, True, 0, L), ws.buf, ws.bytes,
                  stream, flags=0 if r == 0 else reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 0
    expect = hostpools.copy_pools(new_host)
    st = oracle.reshard(old_host, expect, T(*w.old_topo), T(*w.new_topo), L, H, inp.old_tables, inp.new_tables,
                        pairs=pairs)
    for p in pairs:
        assert np.array_equal(staging[p].cpu().numpy(), oracle.staging_buffer(st[p])), f"staging {p}"
    # expand tables B, then try to reuse them for tables A: nothing may be written
    scratch = RankPool.from_host(hostpools.copy_pools(new_host)[0], rank_layers(0, w.new_topo, L),
                                 inp.new_tables.num_blocks, 0)
    plan.unpack(0, window_args(plan, staging, 0, W_old, False, 0, L), scratch.arg, dtb.host, dtb.dev, ws.buf,
                ws.bytes, stream)
    torch.cuda.synchronize()
    assert ws.flag() == 0
    log("[reuse] new tables B expanded; reuse with tables A")
    plan.unpack(0, window_args(plan, staging, 0, W_old, False, 0, L), dst[0].arg, dtn.host, dtn.dev, ws.buf,
                ws.bytes, stream, flags=reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 2
    _unchanged({}, {}, {0: dst[0]}, {0: new_host[0]}, w.elem_bytes)
    # another plan of the same migration does not match this plan's stamps
    plan2 = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    ws.set_flag(0)
    plan2.unpack(0, window_args(plan2, staging, 0, W_old, False, 0, L), dst[0].arg, dtb.host, dtb.dev, ws.buf,
                 ws.bytes, stream, flags=reuse)
    before = {p: b.clone() for p, b in staging.items()}
    plan2.pack(1, src[1].arg, dto.dev, window_args(plan2, staging, 1, W_new, True, 0, L), ws.buf, ws.bytes, stream,
               flags=reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 2
    _unchanged(staging, before, {0: dst[0]}, {0: new_host[0]}, w.elem_bytes)
    # expanding tables A again makes them reusable: every new rank, first call included
    ws.set_flag(0)
    plan.unpack(0, window_args(plan, staging, 0, W_old, False, 0, 0), dst[0].arg, dtn.host, dtn.dev, ws.buf,
                ws.bytes, stream, 0, 0)                                       # empty window: no expansion
    plan.unpack(W_new - 1, window_args(plan, staging, W_new - 1, W_old, False, 0, 1), dst[W_new - 1].arg, dtn.host,
                dtn.dev, ws.buf, ws.bytes, stream, 0, 1)                     # expands, whatever it holds
    for q in range(W_new):
        plan.unpack(q, window_args(plan, staging, q, W_old, False, 0, L), dst[q].arg, dtn.host, dtn.dev, ws.buf,
                    ws.bytes, stream, flags=reuse)
    torch.cuda.synchronize()
    assert ws.flag() == 0
    for q, pool in dst.items():
        got = pool.host(w.elem_bytes)
        for l in expect[q]:
            assert np.array_equal(got[l], expect[q][l]), f"new rank {q} layer {l}"
