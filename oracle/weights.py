"""CPU oracle for the GPU shard rebuild from ReMP's shared weight store (Section 3.3).

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the benchmark
may import or run this module.  It shares no code with the HIP library or its
Python binding and imports neither.

What it computes is the plain definition of a worker's shard under a target
topology (Section 3.3): the pipeline stage decides which layers' tensors the
worker keeps, the tensor rank decides which slice of each partitioned tensor,
and replicated tensors are kept whole.  In NumPy, per tensor: slice every part
the way its split says, then stack the slices along rows.

Readings of points the paper leaves open:

* ranks and layer ownership as for the KV cache: rank(pp, tp) = pp * TP + tp,
  stage p holds equal contiguous layer ranges or an explicit partition;
  tensors outside the decoder layers go to the first stage (token embedding)
  or the last (final norm, LM head);
* a partitioned tensor splits one dimension into `units` equal units; with
  TP <= units tensor rank t keeps units [t*units/TP, (t+1)*units/TP), with
  TP > units (TP a multiple of units, e.g. KV heads under GQA) the single
  unit t*units/TP;
* the splits of a Llama-style decoder are the Megatron ones: Q, K, V, gate,
  up, embedding and LM head split their output rows, the attention output and
  MLP down projections their input columns, norms are replicated;
* fused GPU tensors stack their parts' slices along rows in part order
  (Q | K | V, gate | up);
* Q/K/V biases split by heads like their weights; per-head Q/K norm weights
  and the router of a mixture of experts are replicated; every expert's
  gate / up rows and down columns are split like a dense MLP's.
The split of every part is an input (the model inventory says it); the
oracle applies it by the definition above.

Shapes are elements; every array is [rows][cols] of unsigned integers of the
element width (values are copied, never interpreted).
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from .migration import Topology, pp_owner

REPLICATED, SPLIT_ROWS, SPLIT_COLS = 0, 1, 2
FIRST_STAGE, LAST_STAGE = -1, -2


def units_kept(t: int, tp: int, units: int) -> range:
    """Units of a part split into `units` that tensor rank t keeps (Section 3.3)."""
    if tp <= units:
        if units % tp:
            raise ValueError(f"TP={tp} does not divide units={units}")
        per = units // tp
        return range(t * per, (t + 1) * per)
    if tp % units:
        raise ValueError(f"TP={tp} is not a multiple of units={units}")
    u = t // (tp // units)
    return range(u, u + 1)


def stage_holds(stage: int, layer: int, topo: Topology, L: int) -> bool:
    """Whether pipeline stage `stage` keeps a tensor of `layer` (Section 3.3: PP picks the layers)."""
    if layer == FIRST_STAGE:
        return stage == 0
    if layer == LAST_STAGE:
        return stage == topo.pp - 1
    return pp_owner(layer, topo, L) == stage


def part_slice(a: np.ndarray, split: int, units: int, t: int, tp: int) -> np.ndarray:
    """Tensor rank t's slice of the full part `a` [rows][cols] (Section 3.3: TP slices partitioned tensors)."""
    if split == REPLICATED:
        return a
    kept = units_kept(t, tp, units)
    if split == SPLIT_ROWS:
        per = a.shape[0] // units
        return a[kept.start * per: kept.stop * per, :]
    if split == SPLIT_COLS:
        per = a.shape[1] // units
        return a[:, kept.start * per: kept.stop * per]
    raise ValueError(f"unknown split {split}")


def shard(parts: Sequence[Tuple[np.ndarray, int, int]], t: int, tp: int) -> np.ndarray:
    """Shard of one GPU tensor on tensor rank t: its parts' slices stacked along rows."""
    return np.concatenate([part_slice(a, split, units, t, tp) for (a, split, units) in parts], axis=0)


def rank_shards(tensors: Sequence[Tuple[int, Sequence[Tuple[np.ndarray, int, int]]]], topo: Topology, L: int,
                rank: int) -> Dict[int, np.ndarray]:
    """{tensor index: shard} for every tensor `rank` keeps under `topo`.

    tensors: (layer, [(full part array, split, units), ...]) per GPU tensor.
    """
    stage, t = rank // topo.tp, rank % topo.tp
    return {i: np.ascontiguousarray(shard(parts, t, topo.tp))
            for i, (layer, parts) in enumerate(tensors) if stage_holds(stage, layer, topo, L)}


def shard_shapes(tensors, topo: Topology, L: int, rank: int) -> List[Tuple[int, int]]:
    """Shard shape of every tensor on `rank` ((0, 0) when not kept)."""
    got = rank_shards(tensors, topo, L, rank)
    return [tuple(got[i].shape) if i in got else (0, 0) for i in range(len(tensors))]
