"""A second, element-by-element formulation of the migration, for pinning the oracle.

It shares nothing with the oracle's arithmetic: ownership comes from explicit
rank -> (layers, heads) lists built with numpy.array_split (numpy.repeat for
replicated heads) and found by membership search; paging comes from expanding each table row into its list of
(block, slot) positions; staging is written row by row with a running cursor.
Pure-Python loops, so only for tiny shapes.
"""
from __future__ import annotations

import numpy as np


def explicit_ownership(tp: int, pp: int, L: int, H: int, starts=None):
    """List indexed by global rank id: (layers, heads) that rank holds.

    Ranks are enumerated stage by stage, tensor rank fastest.  With more
    tensor ranks than heads, each head is repeated on consecutive ranks.
    `starts` (stage boundaries) splits the layers at the given points.
    """
    if starts is None:
        stages = [list(map(int, a)) for a in np.array_split(np.arange(L), pp)]
    else:
        stages = [list(map(int, a)) for a in np.split(np.arange(L), list(starts)[1:-1])]
    if tp <= H:
        parts = [list(map(int, a)) for a in np.array_split(np.arange(H), tp)]
    else:
        parts = [[int(h)] for h in np.repeat(np.arange(H), tp // H)]
    out = []
    for p in range(pp):
        for t in range(tp):
            out.append((stages[p], parts[t]))
    return out


def find_rank(own, l: int, h: int) -> int:
    hits = find_ranks(own, l, h)
    assert len(hits) == 1, (l, h, hits)
    return hits[0]


def find_ranks(own, l: int, h: int):
    """Every rank holding (l, h), by membership search."""
    return [i for i, (ls, hs) in enumerate(own) if l in ls and h in hs]


def supplier(own_o, own_n, l: int, h: int, q: int) -> int:
    """Old rank that supplies (l, h) to new rank q: q itself if it holds an old
    replica, else replica number (q's position among the new holders) mod
    (number of old replicas)."""
    cands = find_ranks(own_o, l, h)
    if q in cands:
        return q
    return cands[find_ranks(own_n, l, h).index(q) % len(cands)]


def slot_list(row, block_size: int):
    """Token positions of a table row: token t -> slot_list[t]."""
    out = []
    for b in row:
        for j in range(block_size):
            out.append((int(b), j))
    return out


def migrate(old_pools, new_pools, old_tp, old_pp, new_tp, new_pp, L, H, old_tables, new_tables,
            old_starts=None, new_starts=None):
    """Write every live element of the new ranks present in new_pools."""
    own_o = explicit_ownership(old_tp, old_pp, L, H, old_starts)
    own_n = explicit_ownership(new_tp, new_pp, L, H, new_starts)
    S = len(old_tables.seq_lens)
    for l in range(L):
        for h in range(H):
            for rn in find_ranks(own_n, l, h):
                if rn not in new_pools or l not in new_pools[rn]:
                    continue
                ro = supplier(own_o, own_n, l, h, rn)
                ho = own_o[ro][1].index(h)
                hn = own_n[rn][1].index(h)
                for s in range(S):
                    so = slot_list(old_tables.row(s)[: (int(old_tables.seq_lens[s]) + old_tables.block_size - 1)
                                                      // old_tables.block_size], old_tables.block_size)
                    sn = slot_list(new_tables.row(s)[: (int(new_tables.seq_lens[s]) + new_tables.block_size - 1)
                                                      // new_tables.block_size], new_tables.block_size)
                    for t in range(int(old_tables.seq_lens[s])):
                        bo, jo = so[t]
                        bn, jn = sn[t]
                        for kv in range(2):
                            new_pools[rn][l][kv, bn, jn, hn, :] = old_pools[ro][l][kv, bo, jo, ho, :]


def staging(old_pools, old_tp, old_pp, new_tp, new_pp, L, H, old_tables, old_starts=None, new_starts=None):
    """{(r, q): flat uint8 buffer} for every pair that exchanges at least one row."""
    own_o = explicit_ownership(old_tp, old_pp, L, H, old_starts)
    own_n = explicit_ownership(new_tp, new_pp, L, H, new_starts)
    S = len(old_tables.seq_lens)
    out = {}
    for r in range(len(own_o)):
        for q in range(len(own_n)):
            rows = []
            for l in range(L):
                if l not in own_o[r][0] or l not in own_n[q][0]:
                    continue
                heads = [h for h in range(H) if h in own_o[r][1] and h in own_n[q][1]
                         and supplier(own_o, own_n, l, h, q) == r]
                if not heads:
                    continue
                for kv in range(2):
                    for s in range(S):
                        so = slot_list(old_tables.row(s)[: (int(old_tables.seq_lens[s]) + old_tables.block_size - 1)
                                                          // old_tables.block_size], old_tables.block_size)
                        for t in range(int(old_tables.seq_lens[s])):
                            bo, jo = so[t]
                            for h in heads:
                                ho = own_o[r][1].index(h)
                                rows.append(old_pools[r][l][kv, bo, jo, ho, :].copy())
            if rows:
                out[(r, q)] = np.concatenate([x.reshape(-1).view(np.uint8) for x in rows])
    return out
