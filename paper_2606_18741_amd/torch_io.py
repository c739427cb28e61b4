"""torch plumbing for the C-ABI: device memory, pointers and streams only.

Nothing here touches payload bytes; it allocates buffers with torch and turns
tensors into the addresses libremp_kv.so takes.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence, Tuple

import torch

from . import _lib as rk


class DeviceTables:
    """A host table set and its device mirror (what pack/unpack read on the GPU)."""

    def __init__(self, host: rk.HostTables, device="cuda"):
        self.host = host
        self.lens = torch.from_numpy(host.seq_lens.copy()).to(device)
        self.offs = torch.from_numpy(host.row_offsets.copy()).to(device)
        self.ids = torch.from_numpy(host.block_ids.copy()).to(device)
        self.dev = rk.dev_tables(self.lens, self.offs, self.ids)


def pool_arg(layers: Sequence[Optional[torch.Tensor]], num_blocks: int, layout: int = rk.LAYOUT_NHD) -> rk.PoolArg:
    """PoolArg from one tensor per local layer holding K at [0] and V at [1] in `layout`
    (e.g. [2, num_blocks, block_size, H_loc, head_dim] for NHD)."""
    ks = [None if t is None else t[0] for t in layers]
    vs = [None if t is None else t[1] for t in layers]
    return rk.PoolArg(ks, vs, num_blocks, layout)


def alloc_staging(plan: rk.Plan, pairs, device="cuda",
                  window: Optional[Tuple[int, int]] = None) -> Dict[Tuple[int, int], torch.Tensor]:
    """One uint8 buffer per (src, dst) pair, sized for the layer window (default: all layers)."""
    out = {}
    for (r, q) in pairs:
        nbytes, offs = plan.query(r, q)
        if window is not None:
            nbytes = int(offs[window[1]] - offs[window[0]])
        if nbytes:
            out[(r, q)] = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return out


def staging_args(staging: Dict[Tuple[int, int], torch.Tensor], me: int, world: int, as_src: bool,
                 plan: Optional[rk.Plan] = None, window: Optional[Tuple[int, int]] = None):
    """remp_buffer array by peer rank.

    as_src: entries are staging[(me, q)] for q in range(world) (pack); else
    staging[(r, me)] (unpack).  With plan and window, each entry addresses the
    window's part of a whole-buffer allocation.
    """
    entries = []
    for peer in range(world):
        key = (me, peer) if as_src else (peer, me)
        b = staging.get(key)
        if b is None:
            entries.append(None)
        elif window is None:
            entries.append((b, b.numel()))
        else:
            _, offs = plan.query(*key)
            a, z = int(offs[window[0]]), int(offs[window[1]])
            entries.append(None if z == a else (b.data_ptr() + a, z - a))
    return rk.buffers(entries)


def workspace(plan: rk.Plan, device="cuda") -> torch.Tensor:
    return torch.zeros(plan.workspace_bytes, dtype=torch.uint8, device=device)


def workspace_flag(ws: torch.Tensor) -> int:
    return int(ws[:4].view(torch.int32).item())


def current_stream() -> int:
    return torch.cuda.current_stream().cuda_stream
