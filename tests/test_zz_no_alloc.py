"""The allocation-free unpack (remp_kv_unpack_noalloc) against the workspace unpack (remp_kv_unpack).

remp_kv_unpack_noalloc keeps its scan, descriptor and sort areas in a static
device array of the library instead of a caller workspace.  Its new pools must
equal, byte for byte, what remp_kv_unpack writes from the same staging (and the
oracle's pools), on consecutive calls whose inputs differ in size, with the
status flag delivered to a caller int32 or kept in the array, with
descriptor reuse accepted only for the tables the array last expanded, and
when captured into a HIP graph and replayed.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synthkv

T = oracle.Topology


def _rk():
    import paper_2606_18741_amd as rk
    return rk


def _torch():
    import torch
    return torch


class _Case:
    """One workload: every old rank packed (workspace entry point), staging ready for any new rank."""

    def __init__(self, w):
        import hostpools
        from gpu_harness import DeviceTables, RankPool, Workspace, rank_layers, shape_of, staging_for_pairs, \
            window_args, stream_handle
        rk = _rk()
        self.w = w
        self.inp = synthkv.make_inputs(w)
        L = w.num_layers
        self.plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(self.inp.old_tables))
        self.old_host = hostpools.source_pools(w, self.inp.old_tables)
        self.new_host = hostpools.sentinel_pools(w, self.inp.new_tables)
        self.dto, self.dtn = DeviceTables(self.inp.old_tables), DeviceTables(self.inp.new_tables)
        W_old, W_new = self.plan.info.old_world, self.plan.info.new_world
        self.pairs = [(p.src, p.dst) for p in self.plan.pairs]
        self.staging = staging_for_pairs(self.plan, w.seed, self.pairs)
        self.ws = Workspace(self.plan)
        stream = stream_handle()
        for r in range(W_old):
            src = RankPool.from_host(self.old_host[r], rank_layers(r, w.old_topo, L), self.inp.old_tables.num_blocks,
                                     r)
            self.plan.pack(r, src.arg, self.dto.dev, window_args(self.plan, self.staging, r, W_new, True, 0, L),
                           self.ws.buf, self.ws.bytes, stream)
            _torch().cuda.synchronize()
            assert self.ws.flag() == 0
        self._pool = lambda q: RankPool.from_host(self.new_host[q], rank_layers(q, w.new_topo, L),
                                                  self.inp.new_tables.num_blocks, q)
        self._args = lambda q: window_args(self.plan, self.staging, q, W_old, False, 0, L)
        self._stream = stream
        # the oracle's new pools, from the same sentinel pre-fill
        self.expected = hostpools.copy_pools(self.new_host)
        oracle.reshard(self.old_host, self.expected, T(*w.old_topo), T(*w.new_topo), L, w.num_kv_heads,
                       self.inp.old_tables, self.inp.new_tables)

    def unpack(self, q, noalloc, status=None, flags=0):
        """Fresh sentinel pool of new rank q, unpacked by one entry point; returns the pool."""
        dst = self._pool(q)
        if noalloc:
            self.plan.unpack_noalloc(q, self._args(q), dst.arg, self.dtn.host, self.dtn.dev, status, self._stream,
                                     flags=flags)
        else:
            self.plan.unpack(q, self._args(q), dst.arg, self.dtn.host, self.dtn.dev, self.ws.buf, self.ws.bytes,
                             self._stream, flags=flags)
        _torch().cuda.synchronize()
        return dst


def _status(value):
    torch = _torch()
    return torch.full((1,), value, dtype=torch.int32, device="cuda")


def _same(a, b, what):
    for l in a.store:
        assert _torch().equal(a.store[l], b.store[l]), f"{what}: layer {l} differs"


@pytest.mark.gpu
def test_noalloc_matches_workspace_unpack_on_consecutive_calls():
    """Two calls in a row, the second with a smaller input: each equals remp_kv_unpack's pools and the oracle's."""
    big = synthkv.reduced(synthkv.GQA_70B, num_seqs=9, max_len=700)
    small = synthkv.reduced(synthkv.MHA_7B, num_seqs=3, max_len=90)
    cases = [_Case(big), _Case(small)]
    assert cases[1].plan.workspace_bytes < cases[0].plan.workspace_bytes
    assert cases[1].plan.info.total_tokens < cases[0].plan.info.total_tokens
    for case in cases:
        for q in range(case.plan.info.new_world):
            print(f"[noalloc] {case.w.name} T={case.plan.info.total_tokens} new rank {q}", flush=True)
            ref = case.unpack(q, noalloc=False)
            st = _status(7)
            got = case.unpack(q, noalloc=True, status=st)
            assert int(st.item()) == 0
            _same(ref, got, f"{case.w.name} new rank {q}")
            host = got.host(case.w.elem_bytes)
            for l, want in case.expected[q].items():
                assert np.array_equal(host[l], want), f"{case.w.name} new rank {q} layer {l} differs from the oracle"


@pytest.mark.gpu
def test_noalloc_status_in_scratch_and_descriptor_reuse():
    """status NULL keeps the flag in the static array; reuse works for the tables the array last expanded and is
    refused (status 2, nothing written) after another plan's call."""
    a = _Case(synthkv.reduced(synthkv.GQA_70B_LONG, num_seqs=3, max_len=260))
    b = _Case(synthkv.reduced(synthkv.QWEN3_30B, num_seqs=2, max_len=120))
    q = 0
    ref = a.unpack(q, noalloc=False)
    got = a.unpack(q, noalloc=True, status=None)
    _same(ref, got, "status NULL")
    st = _status(5)
    reused = a.unpack(q, noalloc=True, status=st, flags=_rk().REMP_KV_REUSE_DESCRIPTORS)
    assert int(st.item()) == 5                      # a reusing call leaves the flag as it was
    _same(ref, reused, "reused descriptors")
    b.unpack(q, noalloc=True, status=None)          # another plan expands into the same array
    st = _status(0)
    refused = a.unpack(q, noalloc=True, status=st, flags=_rk().REMP_KV_REUSE_DESCRIPTORS)
    assert int(st.item()) == 2
    fresh = a._pool(q)
    _same(fresh, refused, "refused reuse must write nothing")


def test_noalloc_refuses_plans_beyond_the_scratch():
    """A plan whose workspace exceeds the static array is refused before anything is checked or enqueued."""
    rk = _rk()
    n = 1 << 22                                     # one sequence, 262144 blocks of 16 tokens
    ids = np.arange(n // 16, dtype=np.int32)
    tables = rk.HostTables(np.array([n], np.int32), np.array([0, n // 16], np.int32), ids, n // 16)
    plan = rk.Plan((1, 1), (1, 1), (1, 1, 8, 2, 16, 16), tables)
    assert plan.workspace_bytes > 8 << 20
    with pytest.raises(rk.RempError) as e:
        plan.unpack_noalloc(0, rk.buffers([None]), rk.PoolArg([None], [None], n // 16), tables,
                            rk.dev_tables(None, None, None), None, 0)
    assert e.value.status_name == "REMP_E_SIZE"


@pytest.mark.gpu
def test_noalloc_under_graph_capture():
    """The use the entry point exists for: a no-alloc unpack captured into a HIP graph (after a first call
    outside the capture resolved the device's array) and replayed three times.  Before every replay the
    destination is reset to its sentinel bytes and another plan's no-alloc unpack runs eagerly, overwriting
    the static array; every replay must expand the tables again and equal the oracle, status 0."""
    torch = _torch()
    case = _Case(synthkv.reduced(synthkv.GQA_70B, num_seqs=5, max_len=300))
    other = _Case(synthkv.reduced(synthkv.MHA_7B, num_seqs=2, max_len=80))
    q = 0
    dst = case._pool(q)
    fresh = case._pool(q)
    st = _status(9)

    def run(stream):
        case.plan.unpack_noalloc(q, case._args(q), dst.arg, case.dtn.host, case.dtn.dev, st, stream)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(side.cuda_stream)                       # resolves the device's array outside the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        run(side.cuda_stream)
    torch.cuda.synchronize()
    for rep in range(3):
        for l in dst.store:
            dst.store[l].copy_(fresh.store[l])
        st.fill_(9)
        other.unpack(0, noalloc=True)               # another plan's expansion into the same array
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(st.item()) == 0, f"replay {rep}: status {int(st.item())}"
        host = dst.host(case.w.elem_bytes)
        for l, want in case.expected[q].items():
            assert np.array_equal(host[l], want), f"replay {rep}: layer {l} differs from the oracle"
        print(f"[noalloc] graph replay {rep} matches the oracle", flush=True)
