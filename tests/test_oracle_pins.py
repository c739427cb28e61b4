"""Pins of the CPU oracle against things other than itself.

* two hand-derived worked examples (tests/golden/, derived by hand from the
  definition of Section 3.4.1; the paper prints none);
* identity when the topology and tables do not change;
* TP a->b->a, PP a->b->a and 2-D round trips reproduce the original bytes;
* tag fill: every live (layer, token, head, kv) row appears exactly once in the
  new shards, at the place an independent membership-search formulation
  predicts, and every other byte keeps its sentinel;
* an element-by-element brute force (tests/bruteforce.py) agrees on pools and
  staging;
* a library formulation (concatenate a sequence's blocks in table order and
  truncate) agrees when the block size is unchanged;
* closed-form byte counts of every staging buffer;
* planted mistakes in the oracle make at least one of these pins fail.
"""
from __future__ import annotations

import itertools
import json
import os

import numpy as np
import pytest

import oracle
import oracle.migration as ors
import synthkv
from synthkv import tables_from_rows

import bruteforce
import hostpools

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
T = oracle.Topology


def _divisors(n):
    return [d for d in range(1, n + 1) if n % d == 0]


def _small(L=4, H=4, D=4, bs_o=2, bs_n=2, S=3, max_len=7, old=(2, 1), new=(1, 2), seed=7,
           pool=("slack", 1.5), elem=2):
    w = synthkv.KVWorkload(
        name="pin", num_layers=L, num_kv_heads=H, head_dim=D, elem_bytes=elem, dtype="u16",
        old_block_size=bs_o, new_block_size=bs_n, num_seqs=S, length_law=("uniform", 0, max_len),
        pool_law=pool, old_topo=old, new_topo=new, role="all", seed=seed)
    return w, synthkv.make_inputs(w)


# ---------------------------------------------------------------------------
# hand-derived golden examples
# ---------------------------------------------------------------------------

def _load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        g = json.load(f)
    old_t = tables_from_rows(g["seq_lens"], g["old_rows"], g["old_num_blocks"], g["old_block_size"])
    new_t = tables_from_rows(g["seq_lens"], g["new_rows"], g["new_num_blocks"], g["new_block_size"])
    old_pools = {}
    for key, arr in g["old_pools"].items():
        r, l = map(int, key.split(":"))
        old_pools.setdefault(r, {})[l] = np.array(arr, dtype=np.uint16)
    L, H, D = g["num_layers"], g["num_kv_heads"], g["head_dim"]
    new_topo = T(*g["new_topo"])
    new_pools = {}
    for q in range(new_topo.world):
        for l in oracle.layers_of(q, new_topo, L):
            new_pools.setdefault(q, {})[l] = np.full(
                (2, g["new_num_blocks"], g["new_block_size"], len(oracle.heads_of(q, new_topo, H)), D),
                g["sentinel"], np.uint16)
    return g, old_t, new_t, old_pools, new_pools


GOLDEN_FILES = ["hand_tp2pp1_to_tp1pp2.json", "hand_tp1pp2_to_tp2pp1_reblock.json",
                "hand_replicated_tp4_to_tp2.json"]


@pytest.mark.parametrize("name", GOLDEN_FILES)
def test_golden_hand_example(name):
    g, old_t, new_t, old_pools, new_pools = _load_golden(name)
    L, H = g["num_layers"], g["num_kv_heads"]
    old_topo, new_topo = T(*g["old_topo"]), T(*g["new_topo"])
    pairs = [tuple(map(int, k.split(":"))) for k in g["expected_staging"]]
    stage = oracle.reshard(old_pools, new_pools, old_topo, new_topo, L, H, old_t, new_t, pairs=pairs)
    for key, arr in g["expected_new_pools"].items():
        q, l = map(int, key.split(":"))
        np.testing.assert_array_equal(new_pools[q][l], np.array(arr, dtype=np.uint16), err_msg=key)
    # every new (rank, layer) storage is covered by the fixture
    assert sum(len(d) for d in new_pools.values()) == len(g["expected_new_pools"])
    for key, vals in g["expected_staging"].items():
        r, q = map(int, key.split(":"))
        got = oracle.staging_buffer(stage[(r, q)]).view(np.uint16)
        np.testing.assert_array_equal(got, np.array(vals, dtype=np.uint16), err_msg=key)
    # and no other pair exchanges data
    assert set(oracle.pair_slices(old_topo, new_topo, L, H)) == set(pairs)


# ---------------------------------------------------------------------------
# identity and round trips
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("topo", [(1, 1), (2, 1), (1, 2), (2, 2), (4, 1), (8, 1), (16, 2)])
def test_identity(topo):
    w, inp = _small(old=topo, new=topo)
    old = hostpools.source_pools(w, inp.old_tables)
    new = hostpools.copy_pools(old)
    stage = oracle.reshard(old, new, T(*topo), T(*topo), w.num_layers, w.num_kv_heads,
                           inp.old_tables, inp.old_tables,
                           pairs=[(r, r) for r in range(T(*topo).world)])
    for r in old:
        for l in old[r]:
            np.testing.assert_array_equal(new[r][l], old[r][l])
    # each rank only keeps its own data: pairs are exactly (r, r)
    assert set(oracle.pair_slices(T(*topo), T(*topo), w.num_layers, w.num_kv_heads)) == \
        {(r, r) for r in range(T(*topo).world)}
    assert all(len(v) == len(old[r]) for (r, _), v in stage.items())


def _live_mask(tables, shape_blocks, bs):
    """[nb, bs] boolean: slot holds a live token (by walking tables, not by formula)."""
    m = np.zeros((shape_blocks, bs), dtype=bool)
    for s in range(tables.num_seqs):
        toks = bruteforce.slot_list(tables.row(s)[: (int(tables.seq_lens[s]) + bs - 1) // bs], bs)
        for t in range(int(tables.seq_lens[s])):
            m[toks[t]] = True
    return m


@pytest.mark.parametrize("a,b", [((2, 1), (4, 1)), ((4, 1), (1, 1)), ((1, 2), (1, 4)), ((1, 4), (1, 1)),
                                 ((2, 1), (1, 2)), ((2, 2), (4, 1)), ((1, 4), (4, 1)),
                                 ((2, 1), (8, 1)), ((8, 1), (2, 2)), ((8, 2), (16, 1))])
@pytest.mark.parametrize("reblock", [False, True])
def test_round_trip(a, b, reblock):
    w, inp = _small(old=a, new=b, bs_n=4 if reblock else 2, seed=11)
    L, H = w.num_layers, w.num_kv_heads
    old = hostpools.source_pools(w, inp.old_tables)
    mid = hostpools.sentinel_pools(w, inp.new_tables)
    oracle.reshard(old, mid, T(*a), T(*b), L, H, inp.old_tables, inp.new_tables)
    # back: new->old topology, into a copy of the original pools (the return tables are the originals)
    back = hostpools.copy_pools(old)
    for r in back:
        for l in back[r]:
            back[r][l][...] = 0xDEAD
    oracle.reshard(mid, back, T(*b), T(*a), L, H, inp.new_tables, inp.old_tables)
    live = _live_mask(inp.old_tables, inp.old_tables.num_blocks, inp.old_tables.block_size)
    for r in old:
        for l in old[r]:
            np.testing.assert_array_equal(back[r][l][:, live], old[r][l][:, live])
            assert (back[r][l][:, ~live] == 0xDEAD).all()


# ---------------------------------------------------------------------------
# exactly-once with tags
# ---------------------------------------------------------------------------

MAGIC = 0xA5C3


def _tag_pools(tp, pp, L, H, D, tables, sentinel=0x1234):
    own = bruteforce.explicit_ownership(tp, pp, L, H)
    pools = {}
    for r, (ls, hs) in enumerate(own):
        pools[r] = {}
        for l in ls:
            a = np.full((2, tables.num_blocks, tables.block_size, len(hs), D), sentinel, np.uint16)
            for s in range(tables.num_seqs):
                n = int(tables.seq_lens[s])
                toks = bruteforce.slot_list(tables.row(s)[: (n + tables.block_size - 1) // tables.block_size],
                                            tables.block_size)
                for t in range(n):
                    b, j = toks[t]
                    for i, h in enumerate(hs):
                        for kv in range(2):
                            a[kv, b, j, i, :8] = [MAGIC, s, l, t & 0xFFFF, t >> 16, h, kv, MAGIC ^ 0xFFFF]
            pools[r][l] = a
    return pools


@pytest.mark.parametrize("a,b", [((2, 1), (1, 2)), ((4, 1), (2, 2)), ((1, 4), (2, 1)), ((2, 2), (2, 2)),
                                 ((2, 1), (8, 1)), ((8, 2), (4, 1))])
def test_exactly_once_tags(a, b):
    w, inp = _small(L=4, H=4, D=8, old=a, new=b, bs_o=2, bs_n=4, S=4, max_len=9, seed=5)
    L, H, D = w.num_layers, w.num_kv_heads, w.head_dim
    old = _tag_pools(*a, L, H, D, inp.old_tables)
    new = {}
    own_n = bruteforce.explicit_ownership(*b, L, H)
    for q, (ls, hs) in enumerate(own_n):
        new[q] = {l: np.full((2, inp.new_tables.num_blocks, inp.new_tables.block_size, len(hs), D), 0x7777,
                             np.uint16) for l in ls}
    oracle.reshard(old, new, T(*a), T(*b), L, H, inp.old_tables, inp.new_tables)
    seen = {}
    for q in new:
        for l, arr in new[q].items():
            for kv, blk, slot, hl in itertools.product(range(2), range(arr.shape[1]), range(arr.shape[2]),
                                                       range(arr.shape[3])):
                row = arr[kv, blk, slot, hl]
                if row[0] == MAGIC:
                    assert row[7] == MAGIC ^ 0xFFFF
                    tag = (int(row[1]), int(row[2]), int(row[3]) | (int(row[4]) << 16), int(row[5]), int(row[6]),
                           q)
                    assert tag not in seen, f"row {tag} written twice on rank {q}"
                    seen[tag] = (q, l, blk, slot, hl, kv)
                else:
                    assert (row == 0x7777).all(), "non-live slot modified"
    expect = 0
    for s in range(inp.new_tables.num_seqs):
        n = int(inp.new_tables.seq_lens[s])
        toks = bruteforce.slot_list(inp.new_tables.row(s)[: (n + 3) // 4], 4)
        for l in range(L):
            for h in range(H):
                for q in bruteforce.find_ranks(own_n, l, h):           # every holder gets it once
                    for t in range(n):
                        for kv in range(2):
                            expect += 1
                            blk, slot = toks[t]
                            assert seen[(s, l, t, h, kv, q)] == (q, l, blk, slot, own_n[q][1].index(h), kv)
    assert len(seen) == expect


# ---------------------------------------------------------------------------
# brute force and library formulation
# ---------------------------------------------------------------------------

CASES = [((2, 1), (1, 2), 2, 2), ((1, 2), (2, 1), 2, 4), ((4, 1), (2, 2), 4, 2), ((2, 2), (1, 4), 2, 2),
         ((1, 1), (4, 1), 1, 3), ((2, 2), (4, 1), 4, 8),
         # replicated KV heads (H = 4): TP 8 and 16 hold each head 2 and 4 times
         ((8, 1), (2, 2), 2, 4), ((2, 2), (8, 1), 2, 2), ((8, 1), (8, 1), 2, 2), ((16, 1), (8, 2), 2, 4),
         ((8, 2), (16, 1), 4, 2), ((1, 4), (8, 2), 2, 2),
         # new rank 7 holds head 3 in both topologies: it must keep its own replica, not take old rank 6's
         ((8, 1), (4, 2), 2, 2)]


@pytest.mark.parametrize("a,b,bs_o,bs_n", CASES)
def test_bruteforce_agrees(a, b, bs_o, bs_n):
    w, inp = _small(old=a, new=b, bs_o=bs_o, bs_n=bs_n, S=3, max_len=11, seed=3)
    L, H = w.num_layers, w.num_kv_heads
    # replicas get different bytes so the choice of source replica is visible
    old = hostpools.source_pools(w, inp.old_tables, identical_replicas=False)
    new_o = hostpools.sentinel_pools(w, inp.new_tables)
    new_b = hostpools.copy_pools(new_o)
    pairs = list(oracle.pair_slices(T(*a), T(*b), L, H))
    stage = oracle.reshard(old, new_o, T(*a), T(*b), L, H, inp.old_tables, inp.new_tables, pairs=pairs)
    bruteforce.migrate(old, new_b, *a, *b, L, H, inp.old_tables, inp.new_tables)
    for q in new_o:
        for l in new_o[q]:
            np.testing.assert_array_equal(new_o[q][l], new_b[q][l])
    bst = bruteforce.staging(old, *a, *b, L, H, inp.old_tables)
    assert set(bst) == set(pairs)
    for p in pairs:
        np.testing.assert_array_equal(oracle.staging_buffer(stage[p]), bst[p])


@pytest.mark.parametrize("a,b", [((2, 1), (1, 2)), ((1, 1), (2, 2)), ((4, 1), (1, 4))])
def test_library_formulation(a, b):
    """Same block size: a sequence's logical K (or V) is its blocks, concatenated in
    table order and truncated to its length."""
    w, inp = _small(L=4, H=8, D=4, old=a, new=b, bs_o=4, bs_n=4, S=4, max_len=13, seed=9)
    L, H = w.num_layers, w.num_kv_heads
    old = hostpools.source_pools(w, inp.old_tables)
    new = hostpools.sentinel_pools(w, inp.new_tables)
    oracle.reshard(old, new, T(*a), T(*b), L, H, inp.old_tables, inp.new_tables)
    own_o = bruteforce.explicit_ownership(*a, L, H)
    own_n = bruteforce.explicit_ownership(*b, L, H)
    bs = 4
    for s in range(inp.old_tables.num_seqs):
        n = int(inp.old_tables.seq_lens[s])
        nb = (n + bs - 1) // bs
        for l in range(L):
            # logical [kv, n, H, D] from the old ranks holding layer l
            parts = []
            for r, (ls, hs) in enumerate(own_o):
                if l in ls:
                    blocks = np.take(old[r][l], inp.old_tables.row(s)[:nb], axis=1)   # [2, nb, bs, Hl, D]
                    parts.append((hs[0], blocks.reshape(2, nb * bs, len(hs), -1)[:, :n]))
            logical = np.concatenate([p for _, p in sorted(parts, key=lambda x: x[0])], axis=2)
            for q, (ls, hs) in enumerate(own_n):
                if l in ls:
                    blocks = np.take(new[q][l], inp.new_tables.row(s)[:nb], axis=1)
                    got = blocks.reshape(2, nb * bs, len(hs), -1)[:, :n]
                    np.testing.assert_array_equal(got, logical[:, :, hs[0]:hs[-1] + 1])


# ---------------------------------------------------------------------------
# closed forms and sizes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("L,H", [(4, 8), (12, 12), (80, 8), (40, 40)])
def test_staging_bytes_closed_form(L, H):
    D, e, Tk = 128, 2, 1000
    tps = _divisors(H)[:4] + [2 * H, 4 * H]
    for tp_o, pp_o, tp_n, pp_n in itertools.product(tps, _divisors(L)[:3], tps, _divisors(L)[:3]):
        a, b = T(tp_o, pp_o), T(tp_n, pp_n)
        sb = oracle.staging_bytes(a, b, L, H, D, e, Tk)
        # every new rank receives its whole shard
        hn = H // tp_n if tp_n <= H else 1
        for q in range(b.world):
            assert sum(v for (_, qq), v in sb.items() if qq == q) == 2 * Tk * (L // pp_n) * hn * D * e
        assert sum(sb.values()) == 2 * Tk * L * max(H, tp_n) * D * e
        # without old replication every old rank ships its whole shard, once per new replica of a head
        if tp_o <= H:
            rep_n = max(1, tp_n // H)
            for r in range(a.world):
                assert sum(v for (rr, _), v in sb.items() if rr == r) == \
                    2 * Tk * (L // pp_o) * (H // tp_o) * D * e * rep_n


def test_pair_slices_match_explicit_grouping():
    for L, H in [(4, 4), (6, 12), (8, 8), (4, 2)]:
        tps = _divisors(H) + [2 * H, 4 * H]
        for tp_o, pp_o, tp_n, pp_n in itertools.product(tps, _divisors(L), tps, _divisors(L)):
            own_o = bruteforce.explicit_ownership(tp_o, pp_o, L, H)
            own_n = bruteforce.explicit_ownership(tp_n, pp_n, L, H)
            want = {}
            for q, (ln, hn) in enumerate(own_n):
                for l in ln:
                    for h in hn:
                        r = bruteforce.supplier(own_o, own_n, l, h, q)
                        ls, hs = want.setdefault((r, q), (set(), set()))
                        ls.add(l)
                        hs.add(h)
            want = {k: (sorted(v[0]), sorted(v[1])) for k, v in want.items()}
            assert oracle.pair_slices(T(tp_o, pp_o), T(tp_n, pp_n), L, H) == want


def test_zero_length_sequences_and_empty_population():
    w, inp = _small(S=4, max_len=0)      # every sequence empty
    assert int(inp.lens.sum()) == 0
    old = hostpools.source_pools(w, inp.old_tables)
    new = hostpools.sentinel_pools(w, inp.new_tables)
    ref = hostpools.copy_pools(new)
    pairs = list(oracle.pair_slices(T(2, 1), T(1, 2), w.num_layers, w.num_kv_heads))
    st = oracle.reshard(old, new, T(2, 1), T(1, 2), w.num_layers, w.num_kv_heads, inp.old_tables,
                        inp.new_tables, pairs=pairs)
    for q in new:
        for l in new[q]:
            np.testing.assert_array_equal(new[q][l], ref[q][l])
    for p in pairs:
        assert oracle.staging_buffer(st[p]).size == 0


def test_point_queries_agree_with_reshard():
    w, inp = _small(L=4, H=4, D=4, old=(2, 1), new=(1, 2), bs_o=2, bs_n=4, S=3, max_len=9, seed=13)
    L, H, D = w.num_layers, w.num_kv_heads, w.head_dim
    a, b = T(2, 1), T(1, 2)
    old = hostpools.source_pools(w, inp.old_tables)
    new = hostpools.sentinel_pools(w, inp.new_tables)
    pairs = list(oracle.pair_slices(a, b, L, H))
    st = oracle.reshard(old, new, a, b, L, H, inp.old_tables, inp.new_tables, pairs=pairs)
    bufs = {p: oracle.staging_buffer(st[p]) for p in pairs}
    for s in range(inp.old_tables.num_seqs):
        for t in range(int(inp.lens[s])):
            for l in range(L):
                for h in range(H):
                    r, ob, osl, oh = oracle.old_location(l, h, s, t, a, L, H, inp.old_tables)
                    q, nb, nsl, nh = oracle.new_location(l, h, s, t, b, L, H, inp.new_tables)
                    for kv in range(2):
                        np.testing.assert_array_equal(new[q][l][kv, nb, nsl, nh], old[r][l][kv, ob, osl, oh])
                        off = oracle.staging_location(r, q, l, kv, h, s, t, a, b, L, H, D, 2, inp.lens)
                        np.testing.assert_array_equal(bufs[(r, q)][off:off + 2 * D].view(np.uint16),
                                                      old[r][l][kv, ob, osl, oh])


# ---------------------------------------------------------------------------
# planted mistakes must be caught
# ---------------------------------------------------------------------------

def _pins_pass():
    try:
        for g in GOLDEN_FILES:
            test_golden_hand_example(g)
        test_bruteforce_agrees((4, 1), (2, 2), 4, 2)
        test_bruteforce_agrees((1, 2), (2, 1), 2, 4)
        test_bruteforce_agrees((16, 1), (8, 2), 2, 4)
        test_bruteforce_agrees((8, 1), (4, 2), 2, 2)
        test_round_trip((2, 1), (1, 2), True)
    except Exception:          # a failed assertion or a crash both count as caught
        return False
    return True


def _wrong_rank_of(pp, tp, topo):
    return tp * topo.pp + pp                  # stage-fastest numbering


def _wrong_token_slots(tables, s):
    blk, slot = _orig_token_slots(tables, s)
    return blk, (slot + 1) % int(tables.block_size)   # off-by-one slot


def _wrong_heads_of(r, topo, H):
    rg = _orig_heads_of(r, topo, H)
    return range(rg.start, rg.stop) if topo.tp == 1 else range(rg.start + 1, rg.stop + 1) if rg.stop < H \
        else range(rg.start - 1, rg.stop - 1)


def _wrong_token_offsets(seq_lens):
    off = _orig_token_offsets(seq_lens)
    return np.concatenate([[0], off[:-1]]) if len(off) > 2 else off   # shifted sequence offsets


def _wrong_pp_owner(l, topo, L):
    return l % topo.pp                        # round-robin layers instead of contiguous ranges


def _wrong_tp_owners(h, topo, H):
    return [h % topo.tp] if topo.tp <= H else _orig_tp_owners(h, topo, H)   # round-robin heads


def _swapped_kv_gather(*args, **kw):
    return _orig_gather(*args, **kw)[::-1]    # K and V exchanged


def _wrong_source_first(l, h, q, old, new, L, H):
    cands = ors.holders(l, h, old, L, H)
    return q if q in cands else cands[0]              # always the first replica


def _wrong_source_nolocal(l, h, q, old, new, L, H):
    cands = ors.holders(l, h, old, L, H)
    return cands[ors.holders(l, h, new, L, H).index(q) % len(cands)]    # no local preference


_orig_gather = ors.gather_rows
_orig_tp_owners = ors.tp_owners
_orig_token_slots = ors.token_slots
_orig_heads_of = ors.heads_of
_orig_token_offsets = ors.token_offsets


@pytest.mark.parametrize("target,mutant", [
    ("rank_of", _wrong_rank_of),
    ("token_slots", _wrong_token_slots),
    ("heads_of", _wrong_heads_of),
    ("token_offsets", _wrong_token_offsets),
    ("pp_owner", _wrong_pp_owner),
    ("tp_owners", _wrong_tp_owners),
    ("gather_rows", _swapped_kv_gather),
    ("source_of", _wrong_source_first),
    ("source_of", _wrong_source_nolocal),
])
def test_planted_mistakes_are_caught(monkeypatch, target, mutant):
    assert _pins_pass()
    monkeypatch.setattr(ors, target, mutant)
    assert not _pins_pass(), f"pins did not catch a planted mistake in {target}"


# ---------------------------------------------------------------------------
# physical pool layouts
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("layout", [oracle.NHD, oracle.HND, oracle.ROCM_SPLIT])
@pytest.mark.parametrize("dtype", [np.uint8, np.uint16, np.uint32])
def test_layout_round_trip(layout, dtype):
    rng = np.random.default_rng(4)
    a = rng.integers(0, np.iinfo(dtype).max, size=(2, 5, 8, 3, 32), dtype=dtype)
    np.testing.assert_array_equal(oracle.decode_pool(oracle.encode_pool(a, layout), layout), a)


def test_layout_positions_by_hand():
    """Element (block 1, slot 3, head 2, dim 10) of a fp16 pool with block 4, 3 heads, head_dim 16:
    HND puts it at [1][2][3][10]; the ROCm layout puts K at [1][2][10 // 8][3][10 % 8] and V at
    [1][2][10][3] (x = 16 bytes / 2 = 8 elements)."""
    a = np.zeros((2, 2, 4, 3, 16), dtype=np.uint16)
    a[0, 1, 3, 2, 10] = 0xBEEF
    a[1, 1, 3, 2, 10] = 0xCAFE
    k, v = oracle.encode_pool(a, oracle.HND)
    assert k.shape == (2, 3, 4, 16) and k[1, 2, 3, 10] == 0xBEEF and v[1, 2, 3, 10] == 0xCAFE
    k, v = oracle.encode_pool(a, oracle.ROCM_SPLIT)
    assert k.shape == (2, 3, 2, 4, 8) and v.shape == (2, 3, 16, 4)
    assert k[1, 2, 1, 3, 2] == 0xBEEF and v[1, 2, 10, 3] == 0xCAFE
    assert np.count_nonzero(k) == 1 and np.count_nonzero(v) == 1


# ---------------------------------------------------------------------------
# explicit (uneven) pipeline partitions
# ---------------------------------------------------------------------------

UNEVEN = [((2, 2, (0, 3, 5)), (1, 1, None), 2, 2),
          ((1, 3, (0, 1, 3, 5)), (2, 2, (0, 2, 5)), 2, 4),
          ((2, 1, None), (1, 3, (0, 2, 4, 5)), 4, 2),
          ((8, 2, (0, 4, 5)), (2, 2, (0, 1, 5)), 2, 2)]      # with replicated heads (H = 4)


def _uneven_small(a, b, bs_o, bs_n, seed=17):
    w = synthkv.KVWorkload(name="uneven", num_layers=5, num_kv_heads=4, head_dim=4, elem_bytes=2, dtype="u16",
                           old_block_size=bs_o, new_block_size=bs_n, num_seqs=3, length_law=("uniform", 0, 9),
                           pool_law=("slack", 1.5), old_topo=a, new_topo=b, role="all", seed=seed)
    return w, synthkv.make_inputs(w)


@pytest.mark.parametrize("a,b,bs_o,bs_n", UNEVEN)
def test_uneven_partition_bruteforce(a, b, bs_o, bs_n):
    w, inp = _uneven_small(a, b, bs_o, bs_n)
    L, H = w.num_layers, w.num_kv_heads
    old = hostpools.source_pools(w, inp.old_tables, identical_replicas=False)
    new_o = hostpools.sentinel_pools(w, inp.new_tables)
    new_b = hostpools.copy_pools(new_o)
    pairs = list(oracle.pair_slices(T(*a), T(*b), L, H))
    stage = oracle.reshard(old, new_o, T(*a), T(*b), L, H, inp.old_tables, inp.new_tables, pairs=pairs)
    bruteforce.migrate(old, new_b, a[0], a[1], b[0], b[1], L, H, inp.old_tables, inp.new_tables,
                       old_starts=a[2], new_starts=b[2])
    for q in new_o:
        assert set(new_o[q]) == set(hostpools.rank_layers(q, b[0], b[1], L, b[2]))
        for l in new_o[q]:
            np.testing.assert_array_equal(new_o[q][l], new_b[q][l])
    bst = bruteforce.staging(old, a[0], a[1], b[0], b[1], L, H, inp.old_tables, old_starts=a[2], new_starts=b[2])
    assert set(bst) == set(pairs)
    for p in pairs:
        np.testing.assert_array_equal(oracle.staging_buffer(stage[p]), bst[p])


@pytest.mark.parametrize("a,b,bs_o,bs_n", UNEVEN)
def test_uneven_partition_round_trip(a, b, bs_o, bs_n):
    w, inp = _uneven_small(a, b, bs_o, bs_n, seed=19)
    L, H = w.num_layers, w.num_kv_heads
    old = hostpools.source_pools(w, inp.old_tables)
    mid = hostpools.sentinel_pools(w, inp.new_tables)
    oracle.reshard(old, mid, T(*a), T(*b), L, H, inp.old_tables, inp.new_tables)
    back = hostpools.copy_pools(old)
    for r in back:
        for l in back[r]:
            back[r][l][...] = 0xDEAD
    oracle.reshard(mid, back, T(*b), T(*a), L, H, inp.new_tables, inp.old_tables)
    live = _live_mask(inp.old_tables, inp.old_tables.num_blocks, inp.old_tables.block_size)
    for r in old:
        for l in old[r]:
            np.testing.assert_array_equal(back[r][l][:, live], old[r][l][:, live])


def test_uneven_partition_rejects_bad_bounds():
    for starts in [(0, 5), (1, 3, 5), (0, 3, 3), (0, 4, 6)]:
        with pytest.raises(ValueError):
            oracle.check_divisible(T(1, 2, starts), 5, 4)
