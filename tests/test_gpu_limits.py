"""GPU parity at the library's size limits, byte for byte against the oracle.

The plan takes at most 2^31 - 1 live tokens and fewer than 2^28 live blocks
per block size.  This case holds 2^31 - 2^20 tokens in 2048 sequences and
re-blocks them from 16 to 8 tokens per block, so the new tables hold
2^28 - 2^17 live blocks: token offsets, descriptor counts, sort buckets and
grid sizes all sit just below the bounds the kernels' 32-bit arithmetic
relies on.  One 4-byte head row per token keeps each K or V pool at 8 GiB;
one rank keeps everything (TP1/PP1 on both sides), so the staged path (pack
into the rank's own staging buffer, unpack) and the local fast path both run
the whole cache.  Every byte of the staging buffer and of the new pool
(written by each path in turn) is compared with the oracle, run over
sequence groups on all host cores, and every byte of the source pool is
checked unchanged.  The same configuration passed the CPU model of the
kernels first (tests/test_kernel_model.py, test_model_size_limits).

Needs about 70 GiB of GPU memory and 70 GiB of host memory; about a minute
on MI355X.
"""
from __future__ import annotations

import concurrent.futures
import os
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2606_18741_amd as rk
from paper_2606_18741_amd import torch_io as tio
import synthkv

from edgecases import LIMITS
from gpu_harness import DeviceTables, RankPool, log, shape_of

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

T = oracle.Topology
GROUP = 32           # sequences per oracle task
PIECE = 1 << 30      # bytes per device-to-host comparison


def _sub_tables(t: synthkv.BlockTables, a: int, b: int) -> synthkv.BlockTables:
    """Sequences [a, b) of t as tables of their own (same pool)."""
    o = t.offsets
    return synthkv.BlockTables(t.seq_lens[a:b].copy(), (o[a:b + 1] - o[a]).astype(np.int32),
                               t.ids[o[a]:o[b]].copy(), t.num_blocks, t.block_size)


def _equal_pieces(got: torch.Tensor, want: np.ndarray) -> bool:
    """Every byte of a device tensor against a host array, a piece at a time."""
    g = got.reshape(-1).view(torch.uint8)
    h = torch.from_numpy(np.ascontiguousarray(want).reshape(-1).view(np.uint8))
    if g.numel() != h.numel():
        return False
    for a in range(0, g.numel(), PIECE):
        if not torch.equal(g[a:a + PIECE].cpu(), h[a:a + PIECE]):
            return False
    return True


@pytest.mark.timeout(1500)
def test_size_limits_every_byte():
    torch.cuda.empty_cache()
    t0 = time.time()
    w = LIMITS
    inp = synthkv.make_inputs(w)
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    Tk, n_old, n_new = plan.info.total_tokens, plan.info.old_live_blocks, plan.info.new_live_blocks
    assert Tk == (1 << 31) - (1 << 20) and n_new == (1 << 28) - (1 << 17) and n_old == (1 << 27) - (1 << 16)
    log(f"[limits] T={Tk}, old live blocks {n_old}, new live blocks {n_new}, inputs {time.time() - t0:.0f}s")
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    ws = tio.workspace(plan, "cuda")
    stream = tio.current_stream()
    src = RankPool(w, w.old_topo, inp.old_tables, 0, "source")
    dst = RankPool(w, w.new_topo, inp.new_tables, 0, "sentinel")
    staging = tio.alloc_staging(plan, [(0, 0)], "cuda")
    plan.pack(0, src.arg, dto.dev, tio.staging_args(staging, 0, 1, True), ws, ws.numel(), stream)
    plan.unpack(0, tio.staging_args(staging, 0, 1, False), dst.arg, dtn.host, dtn.dev, ws, ws.numel(), stream)
    torch.cuda.synchronize()
    assert tio.workspace_flag(ws) == 0
    log(f"[limits] staged pack + unpack done ({time.time() - t0:.0f}s)")

    for kv in range(2):                           # the source is unchanged
        ref = torch.empty_like(src.store[0][kv])
        synthkv.fill_pool_layer_(ref, w.seed, 0, 0, kv)
        assert torch.equal(ref, src.store[0][kv]), f"source kv {kv} was modified"
        del ref
    old_h = {0: {0: src.store[0].cpu().numpy()}}
    start = np.empty(tuple(dst.store[0].shape), dtype=old_h[0][0].dtype)
    for kv in range(2):                           # the new pool started from the generator's sentinel bytes
        ref = torch.empty_like(dst.store[0][kv])
        synthkv.fill_sentinel_(ref, w.seed, 0, 0, 0, kv)
        start[kv] = ref.cpu().numpy()
        del ref
    new_h = {0: {0: start}}
    log(f"[limits] host copies ready ({time.time() - t0:.0f}s)")

    # the oracle over groups of sequences (the staging token axis is sequence-major, so group [a, b) owns
    # tokens [tok_off[a], tok_off[b]) of each of K and V); new-pool rows of different groups are disjoint
    tok_off = oracle.token_offsets(inp.lens)
    S = len(inp.lens)
    groups = [(a, min(S, a + GROUP)) for a in range(0, S, GROUP)]
    stage = staging[(0, 0)]
    row = w.num_kv_heads * w.head_dim * w.elem_bytes

    def run(g):
        a, b = g
        part = oracle.reshard(old_h, new_h, T(*w.old_topo), T(*w.new_topo), w.num_layers, w.num_kv_heads,
                              _sub_tables(inp.old_tables, a, b), _sub_tables(inp.new_tables, a, b), layers=[0],
                              pairs=[(0, 0)])
        return g, part[(0, 0)][0]

    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    done = 0
    with concurrent.futures.ThreadPoolExecutor(threads) as ex:
        for (a, b), want in ex.map(run, groups):
            for kv in range(2):
                lo = (kv * Tk + int(tok_off[a])) * row
                hi = (kv * Tk + int(tok_off[b])) * row
                assert _equal_pieces(stage[lo:hi], want[kv]), f"staging kv {kv}, sequences [{a}, {b}) differ"
            done += 1
            if done % 16 == 0:
                log(f"[limits] oracle and staging compared for {done} of {len(groups)} groups "
                    f"({time.time() - t0:.0f}s)")
    assert _equal_pieces(dst.store[0], new_h[0][0]), "new pool (staged path) differs from the oracle"
    log(f"[limits] staged path equals the oracle: {2 * Tk * row} staging bytes, "
        f"{dst.store[0].numel()} new-pool bytes ({time.time() - t0:.0f}s)")
    del staging, stage
    torch.cuda.empty_cache()

    for kv in range(2):                           # the local fast path into a fresh sentinel pool
        synthkv.fill_sentinel_(dst.store[0][kv], w.seed, 0, 0, 0, kv)
    plan.copy_local(0, src.arg, dto.dev, dst.arg, dtn.host, dtn.dev, ws, ws.numel(), stream)
    torch.cuda.synchronize()
    assert tio.workspace_flag(ws) == 0
    assert _equal_pieces(dst.store[0], new_h[0][0]), "new pool (local path) differs from the oracle"
    log(f"[limits] local path equals the oracle ({time.time() - t0:.0f}s)")
    del src, dst, ws, old_h, new_h
    torch.cuda.empty_cache()
