"""A second formulation of the shard rebuild, for pinning the oracle.

It shares nothing with the oracle's arithmetic: which units a tensor rank
keeps comes from explicit lists (numpy.array_split over the unit ids, or
numpy.repeat of the unit ids when there are more ranks than units) found by
position; shards are assembled element by element into Python lists.
Pure-Python loops, so only for tiny shapes.
"""
from __future__ import annotations

import numpy as np

REPLICATED, SPLIT_ROWS, SPLIT_COLS = 0, 1, 2
FIRST_STAGE, LAST_STAGE = -1, -2


def unit_lists(tp: int, units: int):
    """Per tensor rank, the list of unit ids it keeps."""
    if tp <= units:
        return [list(map(int, a)) for a in np.array_split(np.arange(units), tp)]
    return [[int(u)] for u in np.repeat(np.arange(units), tp // units)]


def stage_layers(pp: int, L: int, starts=None):
    if starts is None:
        return [list(map(int, a)) for a in np.array_split(np.arange(L), pp)]
    return [list(map(int, a)) for a in np.split(np.arange(L), list(starts)[1:-1])]


def part_rows(a: np.ndarray, split: int, units: int, t: int, tp: int):
    """The rank's rows of one part, as lists of Python ints."""
    R, C = a.shape
    if split == REPLICATED:
        return [[int(a[r, c]) for c in range(C)] for r in range(R)]
    kept = unit_lists(tp, units)[t]
    if split == SPLIT_ROWS:
        per = R // units
        rows = [u * per + k for u in kept for k in range(per)]
        return [[int(a[r, c]) for c in range(C)] for r in rows]
    per = C // units
    cols = [u * per + k for u in kept for k in range(per)]
    return [[int(a[r, c]) for c in cols] for r in range(R)]


def shards(tensors, tp: int, pp: int, L: int, rank: int, starts=None):
    """{tensor index: 2-D list} for every tensor the rank keeps."""
    stage, t = rank // tp, rank % tp
    mine = stage_layers(pp, L, starts)[stage]
    out = {}
    for i, (layer, parts) in enumerate(tensors):
        held = (layer == FIRST_STAGE and stage == 0) or (layer == LAST_STAGE and stage == pp - 1) or layer in mine
        if not held:
            continue
        rows = []
        for (a, split, units) in parts:
            rows += part_rows(a, split, units, t, tp)
        out[i] = rows
    return out
