"""Seeded synthetic inputs: sequence lengths, paged block tables, pool contents.

This module is shared by the CPU oracle's tests and by the GPU path's tests
and benchmark.  It holds none of the migration's arithmetic: it never decides
which rank owns a layer or a head and never moves a byte between pools.  It
draws

* sequence lengths from a workload's length law,
* block tables by handing out blocks from a shuffled free list (one table set
  per pool, drawn independently for the old and the new pool),
* pool and staging contents as a counter-based hash of (seed, stream id,
  32-bit word index).

The hash is the 32-bit finaliser of MurmurHash3 (Appleby), applied to the word
index XOR a per-stream key.  It is evaluated with torch integer ops on either
device, so a GPU buffer and its CPU counterpart hold the same bytes without a
host->device copy.  Multiplications are split into 16-bit halves so every
intermediate stays below 2**49 in int64 (no reliance on signed overflow).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

from .configs import KVWorkload

_M32 = 0xFFFFFFFF

# stream kinds
SOURCE = 1      # old-pool contents
SENTINEL = 2    # pre-fill of buffers the migration writes into


# ---------------------------------------------------------------------------
# counter-based word generator
# ---------------------------------------------------------------------------

def _fmix32_int(x: int) -> int:
    """MurmurHash3 fmix32 on a Python int (used for key derivation)."""
    x &= _M32
    x ^= x >> 16
    x = (x * 0x85EBCA6B) & _M32
    x ^= x >> 13
    x = (x * 0xC2B2AE35) & _M32
    x ^= x >> 16
    return x


def stream_key(seed: int, *ids: int) -> int:
    """32-bit key of the stream named by (seed, ids...)."""
    k = _fmix32_int(seed * 0x9E3779B1 + 0x7F4A7C15)
    for i in ids:
        k = _fmix32_int(k ^ _fmix32_int((i & _M32) + 0x632BE5AB))
    return k


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2**32 for int64 x in [0, 2**32), without int64 overflow."""
    c_lo, c_hi = c & 0xFFFF, c >> 16
    return (x * c_lo + (((x * c_hi) & 0xFFFF) << 16)) & _M32


def _fmix32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x85EBCA6B)
    x = x ^ (x >> 13)
    x = _mul32(x, 0xC2B2AE35)
    x = x ^ (x >> 16)
    return x


def hash_words(index: torch.Tensor, key: int) -> torch.Tensor:
    """int32 words (two's complement view of the 32-bit hash) at int64 `index`."""
    h = _fmix32((index ^ key) & _M32)
    h = h - ((h >> 31) << 32)           # to signed range before narrowing
    return h.to(torch.int32)


def fill_words_(t: torch.Tensor, seed: int, *stream: int, chunk_words: int = 1 << 26) -> torch.Tensor:
    """Fill contiguous tensor `t` (any dtype, byte size % 4 == 0) in place.

    Word i of the buffer (little-endian 32-bit words) gets hash(i ^ key(seed, stream)).
    """
    assert t.is_contiguous()
    nbytes = t.numel() * t.element_size()
    assert nbytes % 4 == 0, "buffer byte size must be a multiple of 4"
    words = t.view(-1).view(torch.uint8).view(torch.int32)
    key = stream_key(seed, *stream)
    n = words.numel()
    for a in range(0, n, chunk_words):
        b = min(n, a + chunk_words)
        idx = torch.arange(a, b, dtype=torch.int64, device=t.device)
        words[a:b] = hash_words(idx, key)
    return t


def words_at(word_index: np.ndarray, seed: int, *stream: int) -> np.ndarray:
    """The uint32 words that `fill_words_` puts at `word_index` (CPU, any shape)."""
    idx = torch.from_numpy(np.ascontiguousarray(word_index, dtype=np.int64))
    return hash_words(idx, stream_key(seed, *stream)).numpy().view(np.uint32)


def bytes_at(byte_offset: np.ndarray, nbytes: int, seed: int, *stream: int) -> np.ndarray:
    """`nbytes` bytes starting at each byte offset (offsets need not be word aligned).

    Returns uint8 array of shape offsets.shape + (nbytes,).
    """
    off = np.asarray(byte_offset, dtype=np.int64)
    span = off[..., None] + np.arange(nbytes, dtype=np.int64)
    w = words_at(span // 4, seed, *stream)
    return ((w >> (8 * (span % 4)).astype(np.uint32)) & 0xFF).astype(np.uint8)


# ---------------------------------------------------------------------------
# sequence lengths and block tables
# ---------------------------------------------------------------------------

def seq_lens(w: KVWorkload) -> np.ndarray:
    rng = np.random.default_rng([w.seed, 0])
    law = w.length_law
    if law[0] == "uniform":
        lens = rng.integers(law[1], law[2] + 1, size=w.num_seqs)
    elif law[0] == "lognormal":
        median, sigma, cap = law[1], law[2], law[3]
        x = rng.lognormal(mean=math.log(median), sigma=sigma, size=w.num_seqs)
        lens = np.clip(np.rint(x), 1, cap)
    elif law[0] == "fixed":
        lens = np.full(w.num_seqs, law[1])
    else:
        raise ValueError(f"unknown length law {law!r}")
    return lens.astype(np.int32)


@dataclass
class BlockTables:
    """Per-sequence block tables in CSR form (row s = ids[offsets[s]:offsets[s+1]])."""
    seq_lens: np.ndarray     # int32 [S]
    offsets: np.ndarray      # int32 [S+1]
    ids: np.ndarray          # int32 [nnz]
    num_blocks: int          # pool capacity
    block_size: int

    def row(self, s: int) -> np.ndarray:
        return self.ids[self.offsets[s]:self.offsets[s + 1]]

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.shape[0])


def _blocks_needed(lens: np.ndarray, bs: int) -> np.ndarray:
    return (lens.astype(np.int64) + bs - 1) // bs


def make_tables(lens: np.ndarray, block_size: int, pool_law, seed: int, stream: int,
                row_pad: int = 0) -> BlockTables:
    """Hand blocks from a shuffled free list to sequences in order.

    row_pad > 0 appends that many junk ids (-1) to each row, like the unused
    tail of a dense [num_seqs, max_blocks] table; readers must ignore them.
    """
    rng = np.random.default_rng([seed, stream])
    need_per_seq = _blocks_needed(lens, block_size)
    need = int(need_per_seq.sum())
    kind = pool_law[0]
    if kind == "fixed":
        n = int(pool_law[1])
        free = rng.permutation(n)
    elif kind == "slack":
        n = max(1, int(math.ceil(pool_law[1] * need)))
        free = rng.permutation(n)
    elif kind == "fragmented":
        frac = float(pool_law[1])
        n = max(1, int(math.ceil(need / (1.0 - frac))))
        occupied = rng.choice(n, size=int(round(frac * n)), replace=False)
        mask = np.ones(n, dtype=bool)
        mask[occupied] = False
        free = rng.permutation(np.nonzero(mask)[0])
    else:
        raise ValueError(f"unknown pool law {pool_law!r}")
    if need > free.shape[0]:
        raise ValueError(f"pool of {n} blocks cannot hold {need} live blocks")
    rows: List[np.ndarray] = []
    pos = 0
    for k in need_per_seq:
        r = free[pos:pos + k].astype(np.int32)
        pos += int(k)
        if row_pad:
            r = np.concatenate([r, np.full(row_pad, -1, dtype=np.int32)])
        rows.append(r)
    offsets = np.zeros(len(rows) + 1, dtype=np.int32)
    offsets[1:] = np.cumsum([len(r) for r in rows])
    ids = np.concatenate(rows).astype(np.int32) if rows else np.zeros(0, dtype=np.int32)
    return BlockTables(lens.astype(np.int32), offsets, ids, n, block_size)


@dataclass
class Inputs:
    workload: KVWorkload
    lens: np.ndarray
    old_tables: BlockTables
    new_tables: BlockTables


def make_inputs(w: KVWorkload, row_pad: int = 0) -> Inputs:
    lens = seq_lens(w)
    old = make_tables(lens, w.old_block_size, w.pool_law, w.seed, 1, row_pad)
    new = make_tables(lens, w.new_block_size, w.pool_law, w.seed, 2, row_pad)
    return Inputs(w, lens, old, new)


def tables_from_rows(lens: Sequence[int], rows: Sequence[Sequence[int]], num_blocks: int,
                     block_size: int) -> BlockTables:
    lens = np.asarray(lens, dtype=np.int32)
    offsets = np.zeros(len(rows) + 1, dtype=np.int32)
    offsets[1:] = np.cumsum([len(r) for r in rows])
    ids = (np.concatenate([np.asarray(r, dtype=np.int32) for r in rows])
           if len(rows) else np.zeros(0, dtype=np.int32))
    return BlockTables(lens, offsets, ids.astype(np.int32), int(num_blocks), int(block_size))


def torch_dtype_for(elem_bytes: int) -> torch.dtype:
    return {1: torch.uint8, 2: torch.int16, 4: torch.int32}[elem_bytes]


def numpy_dtype_for(elem_bytes: int):
    return {1: np.uint8, 2: np.uint16, 4: np.uint32}[elem_bytes]


def fill_pool_layer_(t: torch.Tensor, seed: int, rank: int, layer: int, kv: int) -> torch.Tensor:
    """Source contents of (old rank, global layer, K=0/V=1) storage."""
    return fill_words_(t, seed, SOURCE, rank, layer, kv)


def fill_sentinel_(t: torch.Tensor, seed: int, *ids: int) -> torch.Tensor:
    return fill_words_(t, seed, SENTINEL, *ids)
