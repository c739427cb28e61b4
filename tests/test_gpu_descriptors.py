"""The block-table expansion and the descriptor sort, read back from the workspace.

A pack expands the old tables (token and block offsets per sequence, one
descriptor {block id, first token, live tokens, sequence} per live block); an
unpack expands the new tables and bucket-sorts their descriptors by physical
block.  These tests read the workspace after each call and compare it with the
same quantities recomputed on the host from their definitions (exclusive
prefix sums, the live part of every table row), for sequence counts around the
scan's 1024-wide chunks, zero-length sequences, padded rows and fragmented
pools; the sorted descriptors must be a permutation of the unsorted ones in
ascending bucket order.  The area offsets follow the documented workspace
layout (header, old and new scans, old and new descriptors, bucket counters,
sorted new descriptors).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import synthkv
from synthkv import tables_from_rows

import kernel_model as km
from gpu_harness import DeviceTables, RankPool, Workspace, log, rank_layers, shape_of, staging_for_pairs, \
    stream_handle, window_args

pytestmark = pytest.mark.gpu


def _tables(lens, bs, rng, pad_max=2, occupied=0.3):
    """Rows of ceil(len / bs) distinct ids from a shuffled pool with some blocks pre-occupied, each row padded
    with 0..pad_max junk ids."""
    need = int(sum((n + bs - 1) // bs for n in lens))
    n_blocks = int(np.ceil(need / (1 - occupied))) + 1
    free = rng.permutation(n_blocks)[:need]
    rows, k = [], 0
    for n in lens:
        nb = (n + bs - 1) // bs
        rows.append(list(free[k:k + nb]) + [-1] * int(rng.integers(0, pad_max + 1)))
        k += nb
    return tables_from_rows(lens, rows, n_blocks, bs)


def _expected(t):
    """Exclusive token and block offsets and the descriptors, from the definitions."""
    lens = t.seq_lens.astype(np.int64)
    bs = t.block_size
    nblk = (lens + bs - 1) // bs
    tok = np.concatenate([[0], np.cumsum(lens)])
    blk = np.concatenate([[0], np.cumsum(nblk)])
    desc = []
    for s in range(len(lens)):
        row = t.row(s)
        for j in range(int(nblk[s])):
            desc.append((int(row[j]), int(tok[s]) + j * bs, int(min(bs, lens[s] - j * bs)), s))
    return tok, blk, np.array(desc, np.int64).reshape(-1, 4)


def _read_i32(ws, off, n):
    return ws[off:off + 4 * n].view(torch.int32).cpu().numpy().astype(np.int64)


def _read_desc(ws, off, n):
    return _read_i32(ws, off, 4 * n).reshape(-1, 4)


CASES = [0, 1, 1023, 1024, 1025, 5000]


@pytest.mark.parametrize("S", CASES)
def test_expansion_and_sort_read_back(S):
    rng = np.random.default_rng(1000 + S)
    lens = rng.integers(0, 50, size=S)
    lens[rng.random(S) < 0.2] = 0                  # zero-length sequences
    if S:
        lens[0] = 37                               # the first sequence always live
    lens = lens.astype(np.int32)
    old_t = _tables(lens, 16, rng)
    new_t = _tables(lens, 32, rng)
    w = synthkv.KVWorkload(name=f"desc{S}", num_layers=1, num_kv_heads=1, head_dim=8, elem_bytes=2, dtype="u16",
                           old_block_size=16, new_block_size=32, num_seqs=S, length_law=("fixed", 0),
                           pool_law=("slack", 1.0), old_topo=(1, 1), new_topo=(1, 1), role="all", seed=S)
    import paper_2606_18741_amd as rk
    plan = rk.Plan((1, 1), (1, 1), shape_of(w), rk.HostTables.of(old_t))
    info = plan.info
    log(f"[descriptors] S={S} T={info.total_tokens} old blocks {info.old_live_blocks} new {info.new_live_blocks}")
    layout = km.workspace_layout(S, info.old_live_blocks, info.new_live_blocks)
    assert layout["total"] == plan.workspace_bytes
    src = RankPool(w, w.old_topo, old_t, 0, "source")
    dst = RankPool(w, w.new_topo, new_t, 0, "sentinel")
    staging = staging_for_pairs(plan, w.seed, [(0, 0)])
    dto, dtn = DeviceTables(old_t), DeviceTables(new_t)
    ws = Workspace(plan)
    plan.pack(0, src.arg, dto.dev, window_args(plan, staging, 0, 1, True, 0, 1), ws.buf, ws.bytes, stream_handle())
    torch.cuda.synchronize()
    tok, blk, desc = _expected(old_t)
    if info.old_live_blocks == 0:                  # nothing to expand: the call returns before any launch
        assert not ws.buf.any().item()
        return
    assert ws.flag() == 0
    assert np.array_equal(_read_i32(ws.buf, layout["scan_old"], S + 1), tok)
    assert np.array_equal(_read_i32(ws.buf, layout["scan_old"] + 4 * (S + 1), S + 1), blk)
    assert np.array_equal(_read_desc(ws.buf, layout["desc_old"], len(desc)), desc)
    assert int(ws.buf[8:16].view(torch.int64).item()) != 0          # the old descriptors' stamp

    plan.unpack(0, window_args(plan, staging, 0, 1, False, 0, 1), dst.arg, dtn.host, dtn.dev, ws.buf, ws.bytes,
                stream_handle())
    torch.cuda.synchronize()
    assert ws.flag() == 0
    tok, blk_n, desc_n = _expected(new_t)
    assert np.array_equal(_read_i32(ws.buf, layout["scan_new"], S + 1), tok)
    assert np.array_equal(_read_i32(ws.buf, layout["scan_new"] + 4 * (S + 1), S + 1), blk_n)
    n = len(desc_n)
    assert np.array_equal(_read_desc(ws.buf, layout["desc_new"], n), desc_n)
    # sort: nb buckets spread over [0, num_blocks); after the scatter each counter is its bucket's end
    nb = (max(n, 1) + 3) // 4
    bucket = np.minimum(desc_n[:, 0] * nb // new_t.num_blocks, nb - 1)
    counts = np.bincount(bucket, minlength=nb)
    assert np.array_equal(_read_i32(ws.buf, layout["bucket_new"], nb), np.cumsum(counts))
    srt = _read_desc(ws.buf, layout["sorted_new"], n)
    sb = np.minimum(srt[:, 0] * nb // new_t.num_blocks, nb - 1)
    assert (np.diff(sb) >= 0).all(), "sorted descriptors out of bucket order"
    key = lambda a: a[np.lexsort(a.T[::-1])]
    assert np.array_equal(key(srt), key(desc_n)), "sorted descriptors are not a permutation of the expansion's"
    assert int(ws.buf[16:24].view(torch.int64).item()) != 0         # the new descriptors' stamp
