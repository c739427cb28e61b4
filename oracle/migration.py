"""CPU oracle for the two-dimensional KV-cache migration of ReMP (Section 3.4).

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import or run this module.  It shares no code with the
HIP library or its Python binding and imports neither.

What it computes is the plain definition the migration has to reach
(Section 3.4.1, logical KV cache model): element KV[l, b, h] held by
rank(l, h, T_old) must end up, unchanged, on rank(l, h, T_new).  The oracle
does not run the paper's plan construction (Algorithm 1); for every
(sequence, layer) it reads each head a new rank needs from the old rank that
supplies it and writes it into the new shard, in NumPy.

Readings of points the paper leaves open:

* ownership: pp_owner(l, PP) = l // (L / PP) (equal contiguous layer ranges,
  L % PP == 0) unless the topology carries an explicit partition (stage p
  holds [starts[p], starts[p+1])), and rank(pp, tp) = pp * TP + tp; heads: with TP <= H
  (H % TP == 0) tensor rank t holds [t*H/TP, (t+1)*H/TP); with TP > H
  (TP % H == 0, GQA replication, allowed by the head-coverage invariant of
  Section 3.4.5) it holds the single head t*H/TP, so each head has TP/H
  replicas;
* source of a head when the old topology replicates it: the destination rank
  itself if it holds a replica (a local copy), else the old replica whose
  index among the head's old replicas is (destination's index among the
  head's new holders) mod (number of old replicas);
* paged storage of a rank: per global layer it owns, K and V arrays of shape
  [num_blocks, block_size, heads it holds, head_dim]; token t of sequence s
  sits in block table[s][t // block_size], slot t % block_size; only live
  tokens (t < n_s) are payload;
* the block mapping across the switch is the caller's new block tables (the
  remapping of block identities that Section 3.4.5 permits); the new block size may
  differ from the old one;
* K and V are two arrays moved identically;
* staging, the contiguous buffer an old rank r fills for a new rank q: the
  (r, q) slices in ascending layer order, each slice laid out as
  [kv][token of all sequences, sequence-major][head of the pair][head_dim].

Array conventions used throughout:
* pools: {rank: {global layer: ndarray [2, num_blocks, block_size, H_loc, D]}}
  (axis 0 is K=0 / V=1), unsigned integers of the element width;
* tables: synthkv.BlockTables (or any object with seq_lens, row(s),
  block_size, num_blocks).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Iterable, List, Optional, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# topology and ownership (Section 3.4.1; replication: Section 3.4.5)
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Topology:
    tp: int
    pp: int
    starts: Optional[Tuple[int, ...]] = None   # explicit stage boundaries [pp + 1], or equal ranges

    @property
    def world(self) -> int:
        return self.tp * self.pp


def check_divisible(topo: Topology, L: int, H: int) -> None:
    if topo.tp < 1 or topo.pp < 1:
        raise ValueError("TP and PP must be positive")
    if topo.starts is not None:
        b = list(topo.starts)
        if len(b) != topo.pp + 1 or b[0] != 0 or b[-1] != L or any(y <= x for x, y in zip(b, b[1:])):
            raise ValueError(f"bad layer partition {b} for L={L}")
    elif L % topo.pp:
        raise ValueError(f"PP={topo.pp} does not divide L={L}")
    if H % topo.tp and topo.tp % H:
        raise ValueError(f"TP={topo.tp} does not fit H={H}")


def stage_bounds(topo: Topology, L: int) -> List[int]:
    """First layer of every stage, then L."""
    if topo.starts is not None:
        return list(topo.starts)
    per = L // topo.pp
    return [p * per for p in range(topo.pp + 1)]


def pp_owner(l: int, topo: Topology, L: int) -> int:
    """Pipeline stage that holds layer l."""
    b = stage_bounds(topo, L)
    return max(p for p in range(topo.pp) if b[p] <= l)


def tp_owners(h: int, topo: Topology, H: int) -> List[int]:
    """Tensor ranks that hold KV head h (one, or TP/H replicas)."""
    if topo.tp <= H:
        return [h // (H // topo.tp)]
    rep = topo.tp // H
    return list(range(h * rep, (h + 1) * rep))


def rank_of(pp: int, tp: int, topo: Topology) -> int:
    """Global rank of (pipeline stage, tensor rank)."""
    return pp * topo.tp + tp


def holders(l: int, h: int, topo: Topology, L: int, H: int) -> List[int]:
    """Global ranks holding (layer l, head h): rank(l, h, T) of Section 3.4.1, as a set."""
    return [rank_of(pp_owner(l, topo, L), t, topo) for t in tp_owners(h, topo, H)]


def source_of(l: int, h: int, q: int, old: Topology, new: Topology, L: int, H: int) -> int:
    """The old rank that supplies (layer l, head h) to new rank q."""
    cands = holders(l, h, old, L, H)
    if q in cands:
        return q
    news = holders(l, h, new, L, H)
    return cands[news.index(q) % len(cands)]


def stage_of_rank(r: int, topo: Topology) -> Tuple[int, int]:
    return r // topo.tp, r % topo.tp


def layers_of(r: int, topo: Topology, L: int) -> range:
    p, _ = stage_of_rank(r, topo)
    b = stage_bounds(topo, L)
    return range(b[p], b[p + 1])


def heads_of(r: int, topo: Topology, H: int) -> range:
    _, t = stage_of_rank(r, topo)
    if topo.tp > H:
        h = t * H // topo.tp
        return range(h, h + 1)
    per = H // topo.tp
    return range(t * per, (t + 1) * per)


def pair_slices(old: Topology, new: Topology, L: int, H: int) -> Dict[Tuple[int, int], Tuple[List[int], List[int]]]:
    """For each (old rank r, new rank q) that exchanges data: (layers, heads).

    By definition: every (l, h) goes to each of its new holders q, from
    source_of(l, h, q); group (l, h) by that (source, holder) pair.
    """
    check_divisible(old, L, H)
    check_divisible(new, L, H)
    groups: Dict[Tuple[int, int], Tuple[set, set]] = {}
    for l in range(L):
        for h in range(H):
            for q in holders(l, h, new, L, H):
                key = (source_of(l, h, q, old, new, L, H), q)
                ls, hs = groups.setdefault(key, (set(), set()))
                ls.add(l)
                hs.add(h)
    return {k: (sorted(v[0]), sorted(v[1])) for k, v in sorted(groups.items())}


def staging_bytes(old: Topology, new: Topology, L: int, H: int, D: int, elem_bytes: int,
                  total_tokens: int) -> Dict[Tuple[int, int], int]:
    """Byte size of every (r, q) staging buffer: all its slices, K and V."""
    out = {}
    for (r, q), (ls, hs) in pair_slices(old, new, L, H).items():
        out[(r, q)] = 2 * total_tokens * len(ls) * len(hs) * D * elem_bytes
    return out


# ---------------------------------------------------------------------------
# paging (where token t of sequence s lives)
# ---------------------------------------------------------------------------

def token_slots(tables, s: int) -> Tuple[np.ndarray, np.ndarray]:
    """(block id, slot) of every live token of sequence s."""
    n = int(tables.seq_lens[s])
    t = np.arange(n, dtype=np.int64)
    bs = int(tables.block_size)
    row = np.asarray(tables.row(s), dtype=np.int64)
    return row[t // bs], t % bs


def token_offsets(seq_lens: np.ndarray) -> np.ndarray:
    """Position of each sequence's first token in the sequence-major token axis."""
    off = np.zeros(len(seq_lens) + 1, dtype=np.int64)
    off[1:] = np.cumsum(np.asarray(seq_lens, dtype=np.int64))
    return off


# ---------------------------------------------------------------------------
# re-shard
# ---------------------------------------------------------------------------

def gather_rows(store: np.ndarray, tables, s: int) -> np.ndarray:
    """Rows of sequence s from one rank's layer storage: [kv, token, local head, D]."""
    blk, slot = token_slots(tables, s)
    return store[:, blk, slot, :, :]


def reshard(old_pools, new_pools, old: Topology, new: Topology, L: int, H: int,
            old_tables, new_tables, layers: Optional[Iterable[int]] = None,
            pairs: Optional[Iterable[Tuple[int, int]]] = None):
    """Re-shard the live KV cache from `old` to `new`.

    old_pools: {old rank: {layer: [2, nb_o, bs_o, H_loc, D]}} -- read only.
    new_pools: {new rank: {layer: [2, nb_n, bs_n, H_loc', D]}} -- written in
               place at live slots only; ranks or layers absent are skipped.
    layers:    global layers to process (default: all).
    pairs:     (old rank, new rank) pairs whose staging to return (default: none).

    Returns {(r, q): {layer: ndarray [2, T, |heads of the pair|, D]}} for the
    requested pairs and processed layers.
    """
    check_divisible(old, L, H)
    check_divisible(new, L, H)
    layers = range(L) if layers is None else sorted(set(layers))
    pairs = [] if pairs is None else sorted(set(pairs))
    S = len(old_tables.seq_lens)
    if list(map(int, old_tables.seq_lens)) != list(map(int, new_tables.seq_lens)):
        raise ValueError("old and new tables must describe the same sequences")
    tok_off = token_offsets(old_tables.seq_lens)
    T = int(tok_off[-1])
    staging: Dict[Tuple[int, int], Dict[int, np.ndarray]] = {p: {} for p in pairs}
    slices = pair_slices(old, new, L, H)
    any_store = next(iter(next(iter(old_pools.values())).values()))
    D, dtype = any_store.shape[-1], any_store.dtype

    for l in layers:
        # (new rank q, head h) <- (old rank r, its local head) for present new ranks
        moves = []
        for q, per_layer in new_pools.items():
            if l in per_layer and l in layers_of(q, new, L):
                for h in heads_of(q, new, H):
                    r = source_of(l, h, q, old, new, L, H)
                    moves.append((q, h - heads_of(q, new, H).start, r, h - heads_of(r, old, H).start))
        cuts = []
        for (r, q) in pairs:
            if (r, q) in slices and l in slices[(r, q)][0]:
                hs = slices[(r, q)][1]
                staging[(r, q)][l] = np.zeros((2, T, len(hs), D), dtype=dtype)
                cuts.append(((r, q), [h - heads_of(r, old, H).start for h in hs]))
        sources = {m[2] for m in moves} | {k[0] for k, _ in cuts}
        if not sources:
            continue
        for s in range(S):
            n = int(old_tables.seq_lens[s])
            if n == 0:
                continue
            rows = {r: gather_rows(old_pools[r][l], old_tables, s) for r in sources}
            nblk, nslot = token_slots(new_tables, s)
            for q, hq, r, hr in moves:
                new_pools[q][l][:, nblk, nslot, hq, :] = rows[r][:, :, hr, :]
            for key, hl in cuts:
                staging[key][l][:, tok_off[s]:tok_off[s] + n, :, :] = rows[key[0]][:, :, hl, :]
    return staging


def staging_buffer(items: Dict[int, np.ndarray]) -> np.ndarray:
    """Concatenate a pair's slices in ascending layer order into one flat buffer."""
    if not items:
        return np.zeros(0, dtype=np.uint8)
    parts = [np.ascontiguousarray(items[l]).reshape(-1).view(np.uint8) for l in sorted(items)]
    return np.concatenate(parts)


# ---------------------------------------------------------------------------
# point queries (for checking sampled rows of very large migrations)
# ---------------------------------------------------------------------------

def old_location(l: int, h: int, s: int, t: int, old: Topology, L: int, H: int, old_tables,
                 new: Optional[Topology] = None, dst: Optional[int] = None):
    """(old rank, block, slot, local head) holding token t of sequence s, layer l, head h.

    With a replicating old topology the supplying replica depends on the
    destination: pass new and dst.
    """
    r = holders(l, h, old, L, H)[0] if dst is None else source_of(l, h, dst, old, new, L, H)
    bs = int(old_tables.block_size)
    blk = int(old_tables.row(s)[t // bs])
    return r, blk, t % bs, h - heads_of(r, old, H).start


def new_location(l: int, h: int, s: int, t: int, new: Topology, L: int, H: int, new_tables, replica: int = 0):
    """(new rank, block, slot, local head) that must hold the same element after the switch."""
    q = holders(l, h, new, L, H)[replica]
    bs = int(new_tables.block_size)
    blk = int(new_tables.row(s)[t // bs])
    return q, blk, t % bs, h - heads_of(q, new, H).start


def staging_location(r: int, q: int, l: int, kv: int, h: int, s: int, t: int, old: Topology,
                     new: Topology, L: int, H: int, D: int, elem_bytes: int, seq_lens,
                     slices=None, tok_off=None) -> int:
    """Byte offset, in the (r, q) staging buffer, of row (l, kv, s, t, h).

    `slices` (pair_slices of the same topologies) and `tok_off` (token_offsets
    of seq_lens) may be passed in to avoid recomputing them per query.
    """
    ps = pair_slices(old, new, L, H) if slices is None else slices
    ls, hs = ps[(r, q)]
    if l not in ls or h not in hs:
        raise ValueError("row is not part of this pair's staging")
    tok_off = token_offsets(seq_lens) if tok_off is None else tok_off
    T = int(tok_off[-1])
    slice_bytes = 2 * T * len(hs) * D * elem_bytes
    row = (kv * T + int(tok_off[s]) + t) * len(hs) + hs.index(h)
    return ls.index(l) * slice_bytes + row * D * elem_bytes


# ---------------------------------------------------------------------------
# physical pool layouts (encodings of the [2, nb, bs, H_loc, D] logical arrays)
# ---------------------------------------------------------------------------

NHD, HND, ROCM_SPLIT = 0, 1, 2


def encode_pool(arr: np.ndarray, layout: int) -> np.ndarray:
    """Physical layout of one rank-layer storage [2 (K, V), nb, bs, H_loc, D].

    NHD: K and V [nb][bs][H][D] (unchanged).  HND: K and V [nb][H][bs][D].
    ROCM_SPLIT (the ROCm paged-attention cache): K [nb][H][D/x][bs][x] with x
    the number of elements in 16 bytes, V [nb][H][D][bs].  Returns a tuple-like
    pair (K array, V array) stacked when shapes agree, else a list.
    """
    k, v = arr[0], arr[1]
    if layout == NHD:
        return [k.copy(), v.copy()]
    if layout == HND:
        return [np.ascontiguousarray(k.transpose(0, 2, 1, 3)), np.ascontiguousarray(v.transpose(0, 2, 1, 3))]
    if layout == ROCM_SPLIT:
        nb, bs, h, d = k.shape
        x = 16 // k.dtype.itemsize
        ks = k.reshape(nb, bs, h, d // x, x).transpose(0, 2, 3, 1, 4)
        vs = v.transpose(0, 2, 3, 1)
        return [np.ascontiguousarray(ks), np.ascontiguousarray(vs)]
    raise ValueError(f"unknown layout {layout}")


def decode_pool(kv, layout: int) -> np.ndarray:
    """Inverse of encode_pool: [2, nb, bs, H_loc, D]."""
    k, v = kv
    if layout == NHD:
        return np.stack([k, v])
    if layout == HND:
        return np.stack([k.transpose(0, 2, 1, 3), v.transpose(0, 2, 1, 3)])
    if layout == ROCM_SPLIT:
        nb, h, dx, bs, x = k.shape
        kk = k.transpose(0, 3, 1, 2, 4).reshape(nb, bs, h, dx * x)
        vv = v.transpose(0, 3, 1, 2)
        return np.stack([kk, vv])
    raise ValueError(f"unknown layout {layout}")
