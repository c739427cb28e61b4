"""GPU parity of the weight-shard rebuild (Section 3.3) against the oracle, through the C-ABI.

Every shard the library builds in HBM from the page-locked host store must
equal, byte for byte, the oracle's slice-and-stack of the same store; bytes
around each shard must stay untouched.  Covered: every rank of many
topologies (replicated KV heads, uneven pipeline partitions), 1-, 2- and
4-byte elements, row lengths that force narrow vectors, tensor windows, grid
caps, both copy engines (gather kernel, DMA), a run beside a KV migration on
another stream, two full Llama3-70B layers plus embedding and LM head, and
the validation errors that must leave memory untouched.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import synthkv
from gpu_harness import DEV, log
from oracle import weights as ow
from oracle.migration import Topology
from weights_harness import abi_tensors, oracle_tensors

pytestmark = pytest.mark.gpu

GUARD = 256          # bytes checked on each side of every shard
SENTINEL = 0xA5


def _rk():
    import paper_2606_18741_amd as rk
    return rk


class Shards:
    """Device buffers for one rank's shards, each with guard bytes on both sides."""

    def __init__(self, plan, rank: int, elem_bytes: int):
        self.bufs = {}
        self.sizes = {}
        for i in range(plan.num_tensors):
            r, c = plan.shard_shape(rank, i)
            if r == 0:
                continue
            n = r * c * elem_bytes
            b = torch.full((n + 2 * GUARD,), SENTINEL, dtype=torch.uint8, device=DEV)
            self.bufs[i] = b
            self.sizes[i] = (r, c, n)

    def dst(self, num_tensors: int):
        return [self.bufs[i][GUARD:].data_ptr() if i in self.bufs else None for i in range(num_tensors)]

    def check(self, want, elem_bytes: int, what: str):
        assert sorted(want) == sorted(self.bufs), what
        for i, b in self.bufs.items():
            r, c, n = self.sizes[i]
            host = b.cpu().numpy()
            assert (host[:GUARD] == SENTINEL).all() and (host[GUARD + n:] == SENTINEL).all(), \
                f"{what}: tensor {i} wrote outside its shard"
            got = host[GUARD:GUARD + n]
            exp = np.ascontiguousarray(want[i]).view(np.uint8).reshape(-1)
            if not np.array_equal(got, exp):
                bad = np.nonzero(got != exp)[0]
                pytest.fail(f"{what}: tensor {i} ({r}x{c}): {bad.size} bytes differ, first at {bad[0]}")


def _topo(t):
    return Topology(t[0], t[1], t[2] if len(t) > 2 else None)


def run_case(spec, topo, flags=0, max_wgs=0, windows=None, ranks=None, store=None, layers=None):
    rk = _rk()
    store = store if store is not None else synthkv.models.host_store(spec, layers, pin=True)
    plan = rk.WeightPlan(topo, spec.num_layers, spec.elem_bytes, abi_tensors(spec, store, layers))
    tensors = oracle_tensors(spec, store, layers)
    stream = torch.cuda.current_stream().cuda_stream
    for rank in (range(plan.world) if ranks is None else ranks):
        log(f"[weights] {spec.name} topo={topo} rank={rank} flags={flags} wgs={max_wgs} windows={windows}")
        sh = Shards(plan, rank, spec.elem_bytes)
        for (a, b) in (windows or [(0, plan.num_tensors)]):
            plan.load(rank, sh.dst(plan.num_tensors), stream, a, b, flags=flags, max_workgroups=max_wgs)
        torch.cuda.synchronize()
        want = ow.rank_shards(tensors, _topo(topo), spec.num_layers, rank)
        sh.check(want, spec.elem_bytes, f"{spec.name} {topo} rank {rank}")
    return plan


TINY_TOPOS = [(1, 1), (2, 1), (4, 1), (8, 1), (2, 2), (4, 2), (8, 4), (2, 2, (0, 3, 4)), (8, 3, (0, 1, 2, 4))]


@pytest.mark.parametrize("topo", TINY_TOPOS)
def test_tiny_all_ranks(topo):
    run_case(synthkv.TINY_DECODER, topo)


@pytest.mark.parametrize("topo", [(1, 1), (2, 2), (8, 1)])
def test_tiny_copy_engine(topo):
    run_case(synthkv.TINY_DECODER, topo, flags=_rk().REMP_W_COPY_ENGINE)


@pytest.mark.parametrize("topo", [(1, 1), (3, 1), (6, 1), (3, 3), (6, 2, (0, 1, 3))])
def test_odd_rows_narrow_vectors(topo):
    run_case(synthkv.ODD_DECODER, topo)


@pytest.mark.parametrize("elem_bytes", [1, 4])
def test_element_sizes(elem_bytes):
    spec = dataclasses.replace(synthkv.TINY_DECODER, name=f"tiny-e{elem_bytes}", elem_bytes=elem_bytes)
    run_case(spec, (4, 2))
    run_case(spec, (8, 1), flags=_rk().REMP_W_COPY_ENGINE)


@pytest.mark.parametrize("spec_name,topo", [("tiny-bias", (2, 2)), ("tiny-bias", (8, 1)), ("tiny-moe", (4, 2)),
                                            ("tiny-moe", (8, 1)), ("tiny-moe", (2, 2, (0, 1, 2)))])
def test_model_variants(spec_name, topo):
    """Q/K/V biases, per-head Q/K norms and mixture-of-experts tensors (hundreds of parts per tensor)."""
    run_case(synthkv.DECODERS[spec_name], topo)
    run_case(synthkv.DECODERS[spec_name], topo, flags=_rk().REMP_W_COPY_ENGINE, ranks=[0])


@pytest.mark.slow
@pytest.mark.parametrize("spec_name,topo,ranks", [("deepseek-r1-distill-qwen-32b", (4, 2), [0, 5]),
                                                  ("qwen3-30b-a3b", (4, 2), [0, 7]),
                                                  ("qwen3-30b-a3b", (8, 1), [6])])
def test_real_shapes_one_layer(spec_name, topo, ranks):
    """Real shapes of the paper's other evaluation models: layer 0 (with its 128 experts for Qwen3-30B-A3B),
    embedding and LM head, whole shards compared."""
    spec = synthkv.DECODERS[spec_name]
    layers = range(1)
    log(f"[weights] filling the {spec.name} store (layer 0, embedding, LM head) in page-locked memory")
    store = synthkv.models.host_store(spec, layers, pin=True, fill_device=DEV)
    run_case(spec, topo, ranks=ranks, store=store, layers=layers)


@pytest.mark.parametrize("max_wgs", [1, 3, 1000])
def test_grid_caps(max_wgs):
    run_case(synthkv.TINY_DECODER, (2, 2), max_wgs=max_wgs)


def test_tensor_windows_match_whole():
    spec = synthkv.TINY_DECODER
    n = len(spec.tensors())
    run_case(spec, (4, 2), windows=[(0, 1), (1, 8), (8, 8), (8, n)])
    run_case(spec, (2, 1), windows=[(0, 5), (5, n)], flags=_rk().REMP_W_COPY_ENGINE)


def test_beside_kv_migration_on_another_stream():
    """A weight load on a second stream while the KV migration runs on the first: both exact."""
    import test_gpu_parity as kv
    rk = _rk()
    spec = dataclasses.replace(synthkv.LLAMA2_7B, num_layers=2)
    store = synthkv.models.host_store(spec, pin=True, fill_device=DEV)
    topo = (2, 1)
    plan = rk.WeightPlan(topo, spec.num_layers, spec.elem_bytes, abi_tensors(spec, store))
    side = torch.cuda.Stream()
    shards = [Shards(plan, r, spec.elem_bytes) for r in range(plan.world)]
    log("[weights] 7B-shaped 2-layer load on a side stream beside the tiny KV migration")
    for r in range(plan.world):
        plan.load(r, shards[r].dst(plan.num_tensors), side.cuda_stream, max_workgroups=32)
    w = synthkv.TINY
    kv.check_against_oracle(w, synthkv.make_inputs(w), log_name="tiny beside weights")
    torch.cuda.synchronize()
    tensors = oracle_tensors(spec, store)
    for r in range(plan.world):
        shards[r].check(ow.rank_shards(tensors, _topo(topo), spec.num_layers, r), spec.elem_bytes, f"7B rank {r}")


@pytest.mark.slow
@pytest.mark.parametrize("topo,ranks", [((4, 2), [0, 3, 7]), ((8, 1), [5])])
def test_llama3_70b_two_layers_full_shards(topo, ranks):
    """Real shapes: layers 0-1, embedding and LM head of Llama3-70B (7.6 GB of store), whole shards compared."""
    spec = synthkv.LLAMA3_70B
    layers = range(2)
    log("[weights] filling the 70B store (layers 0-1, embedding, LM head) in page-locked memory")
    store = synthkv.models.host_store(spec, layers, pin=True, fill_device=DEV)
    run_case(spec, topo, ranks=ranks, store=store, layers=layers)
    run_case(spec, topo, ranks=ranks[:1], store=store, layers=layers, flags=_rk().REMP_W_COPY_ENGINE)


def test_pageable_store_is_refused_and_nothing_written():
    rk = _rk()
    spec = synthkv.TINY_DECODER
    store = synthkv.models.host_store(spec, pin=False)      # ordinary pageable memory
    plan = rk.WeightPlan((2, 1), spec.num_layers, spec.elem_bytes, abi_tensors(spec, store))
    sh = Shards(plan, 0, spec.elem_bytes)
    stream = torch.cuda.current_stream().cuda_stream
    # the DMA flag keeps even a wrongly accepted pageable source fault-free; the check runs either way
    with pytest.raises(rk.RempError) as e:
        plan.load(0, sh.dst(plan.num_tensors), stream, flags=rk.REMP_W_COPY_ENGINE)
    assert e.value.status_name == "REMP_E_INVALID" and "page-locked" in str(e.value)
    torch.cuda.synchronize()
    for b in sh.bufs.values():
        assert (b.cpu().numpy() == SENTINEL).all()
    torch.zeros(4, device=DEV).add_(1)          # no sticky HIP error left behind for the caller
    torch.cuda.synchronize()


def test_host_destination_is_refused():
    rk = _rk()
    spec = synthkv.TINY_DECODER
    store = synthkv.models.host_store(spec, pin=True)
    plan = rk.WeightPlan((1, 1), spec.num_layers, spec.elem_bytes, abi_tensors(spec, store))
    host_dst = torch.full((1 << 20,), SENTINEL, dtype=torch.uint8, pin_memory=True)
    dst = [host_dst.data_ptr()] * plan.num_tensors
    with pytest.raises(rk.RempError) as e:
        plan.load(0, dst, torch.cuda.current_stream().cuda_stream, flags=rk.REMP_W_COPY_ENGINE)
    assert e.value.status_name == "REMP_E_INVALID" and "device memory" in str(e.value)
    torch.cuda.synchronize()
    assert (host_dst.numpy() == SENTINEL).all()
