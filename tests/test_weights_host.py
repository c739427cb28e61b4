"""Host side of the weight-shard rebuild through the C-ABI (no GPU needed):
the library's shard shapes against the oracle's, and every validation error
that is raised before the GPU is touched."""
from __future__ import annotations

import numpy as np
import pytest

import paper_2606_18741_amd as rk
import synthkv
from oracle import weights as ow
from oracle.migration import Topology
from weights_harness import abi_tensors, oracle_tensors

TOPOS = [(1, 1), (2, 1), (4, 1), (8, 1), (2, 2), (4, 2), (8, 4), (1, 4), (2, 2, (0, 3, 4)), (8, 3, (0, 1, 2, 4))]


@pytest.mark.parametrize("topo", TOPOS)
def test_shard_shapes_match_oracle(topo):
    spec = synthkv.TINY_DECODER
    store = synthkv.models.host_store(spec)
    plan = rk.WeightPlan(topo, spec.num_layers, spec.elem_bytes, abi_tensors(spec, store))
    tensors = oracle_tensors(spec, store)
    otopo = Topology(topo[0], topo[1], topo[2] if len(topo) > 2 else None)
    for rank in range(topo[0] * topo[1]):
        want = ow.shard_shapes(tensors, otopo, spec.num_layers, rank)
        got = [plan.shard_shape(rank, i) for i in range(plan.num_tensors)]
        assert got == want, (topo, rank)
        nbytes = sum(r * c for r, c in want) * spec.elem_bytes
        assert plan.shard_bytes(rank) == nbytes
        assert plan.shard_bytes(rank, 1, 3) == sum(r * c for r, c in want[1:3]) * spec.elem_bytes


def test_full_model_shard_bytes_add_up():
    """Closed form: over the ranks of one stage the split parts add up to the whole model
    once, replicated ones once per tensor rank (for TP dividing every split count)."""
    spec = synthkv.LLAMA3_70B
    fake = {p.name: _FakeTensor(0x1000) for p in spec.store_parts()}
    tp, pp = 4, 2
    plan = rk.WeightPlan((tp, pp), spec.num_layers, spec.elem_bytes, abi_tensors(spec, fake))
    total = sum(plan.shard_bytes(r) for r in range(tp * pp))
    parts = spec.store_parts()
    split = sum(p.rows * p.cols for p in parts if p.split != synthkv.models.REPLICATED)
    repl = sum(p.rows * p.cols for p in parts if p.split == synthkv.models.REPLICATED)
    assert total == (split + tp * repl) * spec.elem_bytes
    # new rank 0 of the 70B switch (TP4/PP2): layers 0..39 and the embedding
    h, H, Hkv, D, I, V = spec.hidden, spec.heads, spec.kv_heads, spec.head_dim, spec.intermediate, spec.vocab
    per_layer = ((H + 2 * Hkv) * D * h + h * H * D + 2 * I * h + h * I) // tp + 2 * h
    assert plan.shard_bytes(0) == (40 * per_layer + V * h // tp) * 2


class _FakeTensor:
    """A stand-in host address: planning never dereferences the store."""

    def __init__(self, addr):
        self.addr = addr

    def data_ptr(self):
        return self.addr


def _one(layer=0, rows=8, cols=4, split=rk.REMP_W_SPLIT_ROWS, units=4, host=0x1000):
    return [(layer, [(host, rows, cols, split, units)])]


@pytest.mark.parametrize("topo,num_layers,elem_bytes,tensors,status", [
    ((2, 1), 1, 2, _one(units=3), "REMP_E_INVALID"),                       # units do not divide rows
    ((3, 1), 1, 2, _one(units=4), "REMP_E_INVALID"),                       # TP neither divides nor multiple
    ((2, 1), 1, 2, _one(layer=1), "REMP_E_RANGE"),                         # layer out of range
    ((2, 1), 1, 2, _one(layer=-3), "REMP_E_RANGE"),
    ((2, 1), 1, 2, _one(host=0), "REMP_E_INVALID"),                        # NULL host pointer
    ((2, 1), 1, 2, _one(rows=0), "REMP_E_INVALID"),
    ((2, 1), 1, 2, _one(split=7), "REMP_E_INVALID"),
    ((2, 1), 1, 3, _one(), "REMP_E_INVALID"),                              # elem_bytes
    ((2, 3), 2, 2, _one(), "REMP_E_INVALID"),                              # PP > layers
    ((2, 2), 3, 2, _one(), "REMP_E_UNSUPPORTED"),                          # L % PP without partition
    ((2, 2, (0, 0, 3)), 3, 2, _one(), "REMP_E_INVALID"),                   # empty stage
    ((0, 1), 1, 2, _one(), "REMP_E_INVALID"),
    ((2, 1), 1, 2, [(0, [(0x1000, 8, 4, 1, 4), (0x2000, 8, 6, 1, 4)])], "REMP_E_INVALID"),  # column counts differ
    ((2, 1), 1, 2, [(0, [(0x1000, 8, 4, 2, 4), (0x2000, 8, 4, 1, 4)])], "REMP_E_INVALID"),  # 2 cols vs 4 cols
])
def test_plan_errors(topo, num_layers, elem_bytes, tensors, status):
    with pytest.raises(rk.RempError) as e:
        rk.WeightPlan(topo, num_layers, elem_bytes, tensors)
    assert e.value.status_name == status
    assert rk.remp_last_error()


def test_plan_accepts_empty_model_and_stacked_parts():
    plan = rk.WeightPlan((2, 1), 1, 2, [])
    assert plan.num_tensors == 0 and plan.shard_bytes(1) == 0
    # cols-split part (8 cols / 2 ranks = 4) stacked on a 4-col replicated part
    plan = rk.WeightPlan((2, 1), 1, 2, [(0, [(0x1000, 8, 8, 2, 4), (0x2000, 3, 4, 0, 1)])])
    assert plan.shard_shape(1, 0) == (11, 4)


def test_query_and_load_errors_before_the_gpu():
    plan = rk.WeightPlan((2, 2), 2, 2, _one() + _one(layer=1))
    for args in [(-1, 0), (4, 0), (0, 2), (0, -1)]:
        with pytest.raises(rk.RempError) as e:
            plan.shard_shape(*args)
        assert e.value.status_name == "REMP_E_RANGE"
    with pytest.raises(rk.RempError) as e:
        plan.shard_bytes(0, 1, 3)
    assert e.value.status_name == "REMP_E_RANGE"
    # rank 0 holds tensor 0; a missing destination is rejected before any HIP call
    with pytest.raises(rk.RempError) as e:
        plan.load(0, [None, None], stream=0)
    assert e.value.status_name == "REMP_E_INVALID" and "destination is NULL" in str(e.value)
    for kw, st in [(dict(rank=4), "REMP_E_RANGE"), (dict(tensor_begin=1, tensor_end=0), "REMP_E_RANGE"),
                   (dict(tensor_end=3), "REMP_E_RANGE"), (dict(flags=4), "REMP_E_INVALID"),
                   (dict(max_workgroups=-1), "REMP_E_INVALID")]:
        args = dict(rank=0, dst=[None, None], stream=0)
        args.update(kw)
        with pytest.raises(rk.RempError) as e:
            plan.load(**args)
        assert e.value.status_name == st, kw
    # nothing to do: rank 0 does not hold tensor 1 (layer 1 is on stage 1)
    plan.load(0, [None, None], stream=0, tensor_begin=1, tensor_end=2)
