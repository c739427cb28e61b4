"""GPU-side test harness: device pools, tables and staging buffers for the C-ABI calls.

Pools and staging are torch allocations (plumbing only); every byte the
migration moves is moved by libremp_kv.so.  Contents come from the shared
seeded generator, so the oracle can rebuild the same inputs on the host.
"""
from __future__ import annotations

import sys
from typing import Dict, Iterable, Optional, Tuple

import numpy as np
import torch

import paper_2606_18741_amd as rk
import synthkv
from hostpools import local_heads, source_stream_rank, topo_parts

DEV = "cuda:0"
STAGING_TAG = 99


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def shape_of(w: synthkv.KVWorkload):
    return (w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes, w.old_block_size, w.new_block_size)


class DeviceTables:
    def __init__(self, t: synthkv.BlockTables, device=DEV):
        self.host = rk.HostTables.of(t)
        self.lens = torch.from_numpy(self.host.seq_lens.copy()).to(device)
        self.offs = torch.from_numpy(self.host.row_offsets.copy()).to(device)
        self.ids = torch.from_numpy(self.host.block_ids.copy()).to(device)
        self.dev = rk.dev_tables(self.lens, self.offs, self.ids)


def rank_layers(rank: int, topo, L: int) -> range:
    tp, pp, starts = topo_parts(topo)
    if starts is not None:
        return range(starts[rank // tp], starts[rank // tp + 1])
    per = L // pp
    return range((rank // tp) * per, (rank // tp + 1) * per)


class RankPool:
    """One rank's paged storage: per global layer a [2, nb, bs, H_loc, D] tensor (K, V)."""

    def __init__(self, w: synthkv.KVWorkload, topo, tables: synthkv.BlockTables, rank: int, fill: str,
                 layers: Optional[Iterable[int]] = None, tag: int = 0, device=DEV):
        tp = topo[0]
        self.rank = rank
        self.layers = rank_layers(rank, topo, w.num_layers)
        H_loc = local_heads(w.num_kv_heads, tp)
        dt = synthkv.torch_dtype_for(w.elem_bytes)
        want = set(self.layers if layers is None else layers) & set(self.layers)
        self.store: Dict[int, torch.Tensor] = {}
        for l in self.layers:
            if l not in want:
                continue
            t = torch.empty((2, tables.num_blocks, tables.block_size, H_loc, w.head_dim), dtype=dt, device=device)
            for kv in range(2):
                if fill == "source":
                    synthkv.fill_pool_layer_(t[kv], w.seed, source_stream_rank(rank, tp, w.num_kv_heads), l, kv)
                elif fill == "sentinel":
                    synthkv.fill_sentinel_(t[kv], w.seed, tag, rank, l, kv)
                else:
                    raise ValueError(fill)
            self.store[l] = t
        ks = [self.store[l][0] if l in self.store else None for l in self.layers]
        vs = [self.store[l][1] if l in self.store else None for l in self.layers]
        self.arg = rk.PoolArg(ks, vs, tables.num_blocks)

    @classmethod
    def from_host(cls, arrays: Dict[int, np.ndarray], layers_of_rank: range, num_blocks: int, rank: int,
                  device=DEV) -> "RankPool":
        """Upload host arrays {global layer: [2, nb, bs, H_loc, D]} (unsigned ints of the element width)."""
        self = cls.__new__(cls)
        self.rank = rank
        self.layers = layers_of_rank
        self.store = {}
        for l, a in arrays.items():
            a = np.ascontiguousarray(a)
            signed = {1: np.int8, 2: np.int16, 4: np.int32}[a.dtype.itemsize]
            self.store[l] = torch.from_numpy(a.view(signed)).to(device)
        ks = [self.store[l][0] if l in self.store else None for l in self.layers]
        vs = [self.store[l][1] if l in self.store else None for l in self.layers]
        self.arg = rk.PoolArg(ks, vs, num_blocks)
        return self

    def host(self, elem_bytes: int) -> Dict[int, np.ndarray]:
        nd = synthkv.numpy_dtype_for(elem_bytes)
        return {l: t.cpu().numpy().view(nd) for l, t in self.store.items()}


def staging_for_pairs(plan: rk.Plan, seed: int, pairs: Iterable[Tuple[int, int]], device=DEV,
                      layer_window: Optional[Tuple[int, int]] = None) -> Dict[Tuple[int, int], torch.Tensor]:
    """Sentinel-filled staging per pair, sized for the window (default: all layers)."""
    out = {}
    for (r, q) in pairs:
        nbytes, offs = plan.query(r, q)
        if nbytes == 0:
            continue
        if layer_window is not None:
            nbytes = int(offs[layer_window[1]] - offs[layer_window[0]])
        n = max(nbytes, 4)
        n = (n + 3) // 4 * 4
        buf = torch.empty(n, dtype=torch.uint8, device=device)
        synthkv.fill_sentinel_(buf, seed, STAGING_TAG, r, q)
        out[(r, q)] = buf[:nbytes] if nbytes else buf[:0]
    return out


def staging_args(staging: Dict[Tuple[int, int], torch.Tensor], me: int, world: int, as_src: bool):
    """remp_buffer array by peer rank: as_src -> staging[(me, q)], else staging[(r, me)]."""
    entries = []
    for peer in range(world):
        key = (me, peer) if as_src else (peer, me)
        b = staging.get(key)
        entries.append(None if b is None or b.numel() == 0 else (b, b.numel()))
    return rk.buffers(entries)


class Workspace:
    def __init__(self, plan: rk.Plan, device=DEV):
        self.bytes = plan.workspace_bytes
        self.buf = torch.zeros(self.bytes, dtype=torch.uint8, device=device)

    def flag(self) -> int:
        return int(self.buf[:4].view(torch.int32).item())


def window_args(plan: rk.Plan, staging: Dict[Tuple[int, int], torch.Tensor], me: int, world: int,
                as_src: bool, l0: int, l1: int):
    """remp_buffer array addressing each pair's [l0, l1) window inside its whole staging buffer."""
    entries = []
    for peer in range(world):
        key = (me, peer) if as_src else (peer, me)
        b = staging.get(key)
        if b is None:
            entries.append(None)
            continue
        _, offs = plan.query(*key)
        a, z = int(offs[l0]), int(offs[l1])
        entries.append(None if z == a else (b.data_ptr() + a, z - a))
    return rk.buffers(entries)


def stream_handle() -> int:
    return torch.cuda.current_stream().cuda_stream
