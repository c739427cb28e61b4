"""The CPU model of the kernels (tests/kernel_model.py): bounds, write counts and results.

Every case runs a migration through the model of the library's launch code and
kernels, on the CPU: each load and store is checked against the buffer it must
stay inside, each destination byte must be written at most once, and the bytes
the model moves must equal the oracle's.  The full-size workloads are walked on
sampled workgroups of their real launch shapes (bounds only), and device tables
that disagree with the host ones must be contained.  A planted mistake (the
local copy without its negative-token check) must be caught.
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import oracle
import synthkv

import kernel_model as km
from edgecases import EDGE, LIMITS, SHIFTED_LAYOUTS, shifted_old_lengths_case as _shifted_case
from fuzzcases import layout_cases, layout_count, random_windows, random_workload, seed_range

T = oracle.Topology


def _staged_pairs(m: km.Migration, local: bool):
    return [k for k in m.pairs if not (local and k[0] == k[1])]


def check_model(w, inp=None, windows=None, local=False, lo=km.NHD, ln=km.NHD, wg_bytes=0, seed=0):
    """Run the migration through the model and compare with the oracle; check write counts."""
    inp = inp or synthkv.make_inputs(w)
    m = km.Migration(w, inp, lo, ln, data=True, wg_bytes=wg_bytes, seed=seed)
    flags = m.migrate(windows, local)
    assert all(f == 0 for f in flags), flags
    pairs = _staged_pairs(m, local)
    ref_new = {q: {l: a.copy() for l, a in per.items()} for q, per in m.new_host.items()}
    st = oracle.reshard(m.old_host, ref_new, T(*w.old_topo), T(*w.new_topo), w.num_layers, w.num_kv_heads,
                        inp.old_tables, inp.new_tables, pairs=pairs)
    for k in pairs:
        want = oracle.staging_buffer(st[k])
        reg = m.mem.region(f"stage{k}")
        assert np.array_equal(reg.data, want), f"staging {k} differs from the oracle"
        assert (reg.writes == 1).all(), f"staging {k}: not every byte written exactly once"
    got = m.new_pools()
    for q, per in ref_new.items():
        for l, a in per.items():
            assert np.array_equal(got[q][l], a), f"new rank {q} layer {l} differs from the oracle"
    # the new pools: exactly the live rows written, once; sources never written
    live_rows = _live_rows(inp.new_tables)
    for q, per in ref_new.items():
        for l in per:
            counts = _logical_write_counts(m, q, l)             # [2, nb, bs, H_loc, D]
            per_row = counts.reshape(2, *live_rows.shape, -1)
            assert (per_row[:, live_rows] == 1).all(), f"new rank {q} layer {l}: a live element not written once"
            assert (per_row[:, ~live_rows] == 0).all(), f"new rank {q} layer {l}: a dead slot was written"
    for r in m.old_host:
        for l in m.old_host[r]:
            for kv in range(2):
                assert not m.mem.region(f"o{r}.l{l}.{'KV'[kv]}").writes.any(), "a source pool was written"
    return m


def _logical_write_counts(m: km.Migration, q: int, l: int) -> np.ndarray:
    """Store counts of new rank q's layer l per element, in the logical [2, nb, bs, H_loc, D] order."""
    e = m.eb
    kvs = []
    for kv in range(2):
        wr = m.writes(f"n{q}.l{l}.{'KV'[kv]}").reshape(-1, e)
        assert all(np.array_equal(wr[:, i], wr[:, 0]) for i in range(1, e)), "an element was partly written"
        kvs.append(wr[:, 0].reshape(m.phys[("n", q, l, kv)].shape))
    return oracle.decode_pool(kvs, m.ln)


def _live_rows(tables) -> np.ndarray:
    mask = np.zeros((tables.num_blocks, tables.block_size), bool)
    for s in range(len(tables.seq_lens)):
        blk, slot = oracle.token_slots(tables, s)
        mask[blk, slot] = True
    return mask


# ---------------------------------------------------------------------------
# the workloads (reduced populations), edge cases, windows, local fast path
# ---------------------------------------------------------------------------

REDUCED = ["mha7b", "mha13b", "gqa70b", "gqa70b_long", "qwen30b", "ds32b"]


def test_model_tiny_all_ranks():
    check_model(synthkv.TINY)
    check_model(synthkv.TINY, local=True)


@pytest.mark.parametrize("name", REDUCED)
def test_model_reduced_workloads(name):
    w = synthkv.reduced(synthkv.WORKLOADS[name], num_seqs=3, max_len=120 if name.startswith("gqa") else 60)
    check_model(w)
    check_model(w, local=True)


@pytest.mark.parametrize("name", [n for n in EDGE if n not in ("long_single_sequence", "many_sequences")])
def test_model_edge_cases(name):
    check_model(EDGE[name])
    check_model(EDGE[name], local=True)


def test_model_large_edge_cases():
    """The 20011-token sequence and the 1500 short sequences (staged only: the local copy's prologue is
    the same code on more descriptors)."""
    for name in ("long_single_sequence", "many_sequences"):
        check_model(EDGE[name])


def test_model_padded_rows_and_windows():
    w = EDGE["uneven_pp"]
    check_model(w, inp=synthkv.make_inputs(w, row_pad=3))
    w2 = synthkv.reduced(synthkv.GQA_70B_LONG, num_seqs=2, max_len=100)
    check_model(w2, windows=[(0, 1), (1, 7), (7, 40), (40, 41), (41, 80)])
    check_model(w2, windows=[(0, 13), (13, 80)], local=True)


@pytest.mark.parametrize("wg_bytes", [2048, 8192, 32768, 262144, 1 << 20])
def test_model_workgroup_sizes(wg_bytes):
    """The tuning override changes launch shapes only: every shape stays in bounds and moves the same bytes."""
    for w in (synthkv.reduced(synthkv.MHA_7B, num_seqs=2, max_len=40).replace(num_layers=8),
              synthkv.reduced(synthkv.GQA_70B, num_seqs=2, max_len=60).replace(num_layers=16),
              EDGE["merged_rows_mha"]):
        check_model(w, wg_bytes=wg_bytes)
        check_model(w, wg_bytes=wg_bytes, local=True)


# ---------------------------------------------------------------------------
# pool layouts (head tiles through LDS)
# ---------------------------------------------------------------------------

LAYOUT_PAIRS = [(0, 1), (1, 0), (0, 2), (2, 0), (2, 2), (1, 2), (2, 1), (1, 1)]


def _layout_shapes():
    base = dict(name="lay", num_layers=4, num_kv_heads=8, head_dim=64, elem_bytes=2, dtype="u16",
                old_block_size=16, new_block_size=16, num_seqs=3, length_law=("uniform", 0, 70),
                pool_law=("slack", 1.3), old_topo=(2, 1), new_topo=(1, 2), role="all", seed=31)
    out = []
    for c in (dict(), dict(old_block_size=16, new_block_size=32, old_topo=(4, 1), new_topo=(2, 2)),
              dict(elem_bytes=1, head_dim=32, old_block_size=16, new_block_size=32),
              dict(elem_bytes=4, head_dim=16, old_block_size=8, new_block_size=4),
              dict(num_kv_heads=4, old_topo=(8, 1), new_topo=(2, 2)),
              dict(num_kv_heads=8, head_dim=128, old_topo=(8, 1), new_topo=(4, 2))):
        kw = dict(base)
        kw.update(c)
        out.append(synthkv.KVWorkload(**kw))
    return out


@pytest.mark.parametrize("lo,ln", LAYOUT_PAIRS)
def test_model_layouts(lo, ln):
    for w in _layout_shapes():
        if ((w.old_block_size * w.elem_bytes) % 16 and lo == 2) or ((w.new_block_size * w.elem_bytes) % 16 and ln == 2):
            continue
        check_model(w, lo=lo, ln=ln)
        check_model(w, lo=lo, ln=ln, local=True)


# ---------------------------------------------------------------------------
# seeded random configurations (the GPU fuzz generator)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", seed_range(40))
def test_model_fuzz(seed):
    w = random_workload(seed)
    inp = synthkv.make_inputs(w)
    check_model(w, inp, windows=random_windows(seed, w.num_layers), seed=seed)
    check_model(w, inp, local=True, seed=seed)


@pytest.mark.parametrize("seed,lo,ln", layout_cases(layout_count(20)))
def test_model_fuzz_layouts(seed, lo, ln):
    w = random_workload(seed)
    inp = synthkv.make_inputs(w)
    check_model(w, inp, lo=lo, ln=ln, seed=seed)
    check_model(w, inp, lo=lo, ln=ln, local=True, seed=seed)


# ---------------------------------------------------------------------------
# full-size launch shapes: grid order, chunk coverage, sampled workgroups in bounds
# ---------------------------------------------------------------------------

def _coverage(launch: km.Launch, n_desc: int) -> None:
    """The cell order is a bijection of the grid, and the workgroups of each slice cover its 2 * n_desc
    (block, K/V) units exactly once."""
    gx, gy = launch.grid
    cx, cy = km.grid_cells(gx, gy, launch.xcd)
    assert np.unique(cy * gx + cx).size == gx * gy
    C = launch.args["C"]
    units = 2 * n_desc
    assert (gx - 1) * C < units <= gx * C
    assert C <= km.MAX_UNITS_PER_WG


@pytest.mark.parametrize("name", REDUCED)
def test_model_full_size_launch_shapes(name):
    w = synthkv.WORKLOADS[name]
    inp = synthkv.make_inputs(w)
    m = km.Migration(w, inp, data=False, seed=7)
    ro, qn = w.role
    launches = m.pack_launches(ro, 0, w.num_layers)
    assert launches
    for Lc in launches:
        if Lc.kernel in ("copy_slices", "copy_rows"):
            _coverage(Lc, m.n_old)
    assert m.pack(ro, sample=48) == 0
    launches = m.unpack_launches(qn, 0, w.num_layers)
    for Lc in launches:
        if Lc.kernel in ("copy_slices", "copy_rows"):
            _coverage(Lc, m.n_new)
    assert m.unpack(qn, sample=48) == 0
    if (ro, qn) in m.pairs and ro == qn:
        for Lc in m.local_launches(ro, 0, w.num_layers):
            _coverage(Lc, m.n_new)
        assert m.copy_local(ro, sample=48) == 0


@pytest.mark.skipif(not os.environ.get("REMP_MODEL_LIMITS"),
                    reason="about 25 minutes and 40 GiB of host memory: set REMP_MODEL_LIMITS=1")
def test_model_size_limits():
    """The size-limit case of the GPU suite (2^31 - 2^20 tokens, 2^28 - 2^17 new live blocks): the whole
    expansion and descriptor sort of both sides, then sampled workgroups of every pack, unpack and local-copy
    launch, bounds and exactly-once writes checked."""
    w = LIMITS
    m = km.Migration(w, synthkv.make_inputs(w), data=False, seed=3)
    assert m.T == (1 << 31) - (1 << 20) and m.n_new == (1 << 28) - (1 << 17)
    assert m.pack(0, sample=64) == 0
    assert m.unpack(0, sample=64) == 0
    assert m.copy_local(0, sample=64) == 0


@pytest.mark.parametrize("lo,ln", [(1, 1), (2, 2), (0, 2), (1, 0)])
def test_model_full_size_layouts(lo, ln):
    w = synthkv.GQA_70B
    m = km.Migration(w, synthkv.make_inputs(w), lo, ln, data=False, seed=9)
    assert m.pack(0, sample=24) == 0
    assert m.unpack(0, sample=24) == 0
    assert m.copy_local(0, sample=24) == 0


# ---------------------------------------------------------------------------
# device tables that disagree with the host tables
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("lo,ln,bn", SHIFTED_LAYOUTS)
def test_model_shifted_old_lengths_are_contained(lo, ln, bn):
    """The local copies combine the new expansion's token offsets with the old one's; old device lengths
    that shift a sequence start (same total) must neither leave the pools nor go unreported."""
    w, inp, dev_old = _shifted_case(bn)
    m = km.Migration(w, inp, lo, ln, data=True, dev_old=dev_old)
    flags = [m.copy_local(r) for r in range(min(m.old.tp * m.old.pp, m.new.tp * m.new.pp))]
    assert all(f == 1 for f in flags), f"shifted device lengths went unreported: {flags}"


def test_model_out_of_range_ids_are_contained():
    w = synthkv.reduced(synthkv.TINY, num_seqs=3, max_len=60)
    inp = synthkv.make_inputs(w)
    t = inp.old_tables
    dev_old = (t.seq_lens, t.offsets, np.full_like(t.ids, 1 << 30))
    m = km.Migration(w, inp, data=True, dev_old=dev_old)
    assert m.pack(0) == 1
    for k in m.pairs:
        assert not m.mem.region(f"stage{k}").writes.any(), "a pack with out-of-range ids copied something"


def test_model_catches_the_planted_negative_token_mistake(monkeypatch):
    """Without the check that a row's token index is not negative, the shifted lengths make the local copy
    read before an old block: the model must fail."""
    w, inp, dev_old = _shifted_case()

    def without_check(mem, d, rows, tok_off_addr, blk_off_addr, old_desc_addr, n_old, bo):
        live = rows < d[:, 2]
        seq = d[:, 3]
        t_ = np.zeros(len(d), np.int64)
        ob = np.zeros(len(d), np.int64)
        slot = np.zeros(len(d), np.int64)
        if live.any():
            to = mem.load_i32(tok_off_addr, seq[live], "copy_local: token offsets")
            b_ = mem.load_i32(blk_off_addr, seq[live], "copy_local: old block offsets")
            t_[live] = d[live, 1] - to + rows[live]
            q = km.cdiv_trunc(t_[live], bo)
            ob[live] = b_ + q
            slot[live] = t_[live] - q * bo
        ok = live & (ob >= 0) & (ob < n_old)             # planted: no t >= 0
        od = np.zeros((len(d), 4), np.int64)
        if ok.any():
            od[ok] = km._desc_load(mem, old_desc_addr, ob[ok], "copy_local: old descriptors")
        ok &= (od[:, 3] == seq) & (slot < od[:, 2])
        return ok, od, slot, bool((live & ~ok).any())

    monkeypatch.setattr(km, "_resolve_rows", without_check)
    m = km.Migration(w, inp, data=True, dev_old=dev_old)
    with pytest.raises(km.ModelError):
        for r in range(min(m.old.tp * m.old.pp, m.new.tp * m.new.pp)):
            m.copy_local(r)


def test_flag_reads_check():
    """The check of the local tile copy's source-flag reads accepts the word groups every ROCm V vector
    reads (block sizes that are multiples of the vector's elements) and rejects a group that is
    misaligned or runs past its tile's rows."""
    for bn, m, T in ((16, 8, 4), (32, 16, 2), (8, 4, 7), (64, 8, 1)):
        lrow = 16 * 17
        s0 = np.arange(0, bn, m)
        tiles = np.repeat(np.arange(T), s0.size)
        km._check_flag_reads(T, bn, lrow, tiles, np.tile(s0, T), m, "ok")
    with pytest.raises(km.ModelError):
        km._check_flag_reads(4, 16, 272, np.array([1]), np.array([4]), 8, "misaligned")
    with pytest.raises(km.ModelError):
        km._check_flag_reads(4, 12, 272, np.array([0]), np.array([8]), 8, "past the tile")
