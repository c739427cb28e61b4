"""Seeded random configurations through the GPU path, bit-exact against the oracle.

Shapes, element sizes (1, 2, 4 bytes), head counts with and without
replication, even and explicit uneven pipeline partitions, block sizes that
change across the switch, empty and fragmented pools, and layer windows are
drawn at random (tests/fuzzcases.py); every case runs the staged path over
random layer windows and the local fast path, and (half the seeds each)
the staged or the local path over random windows with the block
descriptors expanded once and reused by every later call.  A second set
of seeds runs on HND and ROCm pools (random layout pairs), staged and local.
"""
from __future__ import annotations

import pytest

import synthkv
from fuzzcases import layout_cases, layout_count, random_windows, random_workload, seed_range
from test_gpu_parity import _layouts_case, _local_layouts_case, check_against_oracle

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", seed_range(40))
def test_random_configuration(seed):
    w = random_workload(seed)
    inp = synthkv.make_inputs(w)
    check_against_oracle(w, inp, windows=random_windows(seed, w.num_layers),
                         log_name=f"fuzz{seed} L{w.num_layers} H{w.num_kv_heads} D{w.head_dim} e{w.elem_bytes} "
                                  f"{w.old_topo}->{w.new_topo} bs {w.old_block_size}->{w.new_block_size}")
    check_against_oracle(w, inp, local=True, log_name=f"fuzz{seed} local")
    check_against_oracle(w, inp, windows=random_windows(seed + 1000, w.num_layers), local=bool(seed % 2),
                         reuse=True, log_name=f"fuzz{seed} reuse")


@pytest.mark.parametrize("seed,lo,ln", layout_cases(layout_count(20)))
def test_random_configuration_layouts(seed, lo, ln):
    w = random_workload(seed)
    _layouts_case(w, lo, ln, reuse=bool(seed % 2))
    _local_layouts_case(w, lo, ln, reuse=seed % 3 == 0)
