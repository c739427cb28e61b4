"""Host-side (NumPy) pools filled from the shared seeded generator.

Test harness code: builds the {rank: {layer: [2, nb, bs, H_loc, D]}} arrays the
oracle reads and writes, with the same bytes the GPU tests put in HBM.
"""
from __future__ import annotations

import numpy as np
import torch

import synthkv


def local_heads(H: int, tp: int) -> int:
    return H // tp if tp <= H else 1


def source_stream_rank(r: int, tp: int, H: int) -> int:
    """Stream id of old rank r's contents: replicas of the same head (TP > H)
    share the lowest replica's stream, so they hold identical bytes."""
    if tp <= H:
        return r
    rep = tp // H
    return r - (r % tp) % rep


def topo_parts(topo):
    """(tp, pp, starts or None) from a (tp, pp) or (tp, pp, starts) topology tuple."""
    return int(topo[0]), int(topo[1]), (tuple(topo[2]) if len(topo) > 2 and topo[2] is not None else None)


def rank_layers(r: int, tp: int, pp: int, L: int, starts=None):
    p = r // tp
    if starts is not None:
        return range(starts[p], starts[p + 1])
    per = L // pp
    return range(p * per, (p + 1) * per)


def source_pools(w: synthkv.KVWorkload, tables, ranks=None, layers=None, identical_replicas=True):
    """Old-pool contents for the given old ranks (default: all) and layers.

    identical_replicas=False gives every replica its own bytes (to see which
    replica a head was taken from).
    """
    tp, pp, starts = topo_parts(w.old_topo)
    H_loc = local_heads(w.num_kv_heads, tp)
    dt = synthkv.torch_dtype_for(w.elem_bytes)
    out = {}
    for r in (range(tp * pp) if ranks is None else ranks):
        out[r] = {}
        for l in rank_layers(r, tp, pp, w.num_layers, starts):
            if layers is not None and l not in layers:
                continue
            t = torch.empty((2, tables.num_blocks, tables.block_size, H_loc, w.head_dim), dtype=dt)
            key = source_stream_rank(r, tp, w.num_kv_heads) if identical_replicas else r
            for kv in range(2):
                synthkv.fill_pool_layer_(t[kv], w.seed, key, l, kv)
            out[r][l] = t.numpy().view(synthkv.numpy_dtype_for(w.elem_bytes))
    return out


def sentinel_pools(w: synthkv.KVWorkload, tables, ranks=None, layers=None, tag: int = 0):
    """New-pool pre-fill (sentinel stream) for the given new ranks."""
    tp, pp, starts = topo_parts(w.new_topo)
    H_loc = local_heads(w.num_kv_heads, tp)
    dt = synthkv.torch_dtype_for(w.elem_bytes)
    out = {}
    for q in (range(tp * pp) if ranks is None else ranks):
        out[q] = {}
        for l in rank_layers(q, tp, pp, w.num_layers, starts):
            if layers is not None and l not in layers:
                continue
            t = torch.empty((2, tables.num_blocks, tables.block_size, H_loc, w.head_dim), dtype=dt)
            for kv in range(2):
                synthkv.fill_sentinel_(t[kv], w.seed, tag, q, l, kv)
            out[q][l] = t.numpy().view(synthkv.numpy_dtype_for(w.elem_bytes))
    return out


def copy_pools(pools):
    return {r: {l: a.copy() for l, a in d.items()} for r, d in pools.items()}


def element_offsets(layout: int, kv: int, blk, slot, hl, d, H_loc: int, bs: int, D: int, elem_bytes: int):
    """Element index, inside one layer's K or V storage in `layout`, of element (block, slot, local head, dim).

    NHD [nb][bs][H][D]; HND [nb][H][bs][D]; ROCm split: K [nb][H][D/x][bs][x] (x = elements in 16 bytes),
    V [nb][H][D][bs].  Arguments broadcast (NumPy int64)."""
    blk, slot, hl, d = (np.asarray(a, dtype=np.int64) for a in (blk, slot, hl, d))
    if layout == 0:
        return ((blk * bs + slot) * H_loc + hl) * D + d
    if layout == 1:
        return ((blk * H_loc + hl) * bs + slot) * D + d
    x = 16 // elem_bytes
    if kv == 0:
        return (((blk * H_loc + hl) * (D // x) + d // x) * bs + slot) * x + d % x
    return ((blk * H_loc + hl) * D + d) * bs + slot
