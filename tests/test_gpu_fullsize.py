"""GPU parity at the workloads' full sizes, in the launch configuration the benchmark times.

The GPU plays old rank r0 (packs everything it sends) and new rank q0 (unpacks
everything it receives); the staging other old ranks send to q0 is packed by
the same library from their own generated pools.  Large workloads run in layer
windows (the paper's layer-wise streaming) to bound memory, expanding the
block tables in the first pack and unpack only and reusing the descriptors in
every later call; the 70B GQA share runs as one window, exactly like the
benchmark.

Checked against the oracle:
* sampled staging rows and sampled new-pool rows (uniform over tokens, plus the
  first and last token of every sequence), whose expected bytes the oracle's
  point queries locate in the generated source pools;
* properties over every byte: the new pool differs from its sentinel pre-fill
  at exactly the live (block, slot) rows of the new tables, and the source
  pools are unchanged.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_18741_amd as rk
from paper_2606_18741_amd import torch_io as tio
import synthkv

from gpu_harness import DeviceTables, RankPool, log, shape_of
from hostpools import element_offsets, local_heads

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

T = oracle.Topology
FULL = {
    "mha7b": None,          # one window
    "mha13b": 20,           # layers per window
    "gqa70b": None,
    "gqa70b_long": 20,
    "qwen30b": None,
    "ds32b": 16,
}


def _sample_tokens(rng, lens, n):
    """(seq, token) pairs: n uniform over all tokens, plus first and last token of every sequence."""
    tok_off = oracle.token_offsets(lens)
    Tk = int(tok_off[-1])
    u = rng.integers(0, Tk, size=n)
    s = np.searchsorted(tok_off, u, side="right") - 1
    t = u - tok_off[s]
    extra_s, extra_t = [], []
    for q, ln in enumerate(lens):
        if ln > 0:
            extra_s += [q, q]
            extra_t += [0, int(ln) - 1]
    return np.concatenate([s, extra_s]).astype(np.int64), np.concatenate([t, extra_t]).astype(np.int64)


def _source_bytes(w, old_topo, old_tables, l, kv, h, s, t, layout=0):
    """Expected bytes of (layer l, kv, head h, seq s, token t) from the generated source pools, whose
    storage the library reads in `layout`."""
    L, H, D, e = w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes
    H_loc = local_heads(H, old_topo.tp)
    bs = old_tables.block_size
    out = np.empty((len(l), D * e), np.uint8)
    groups = {}
    for i in range(len(l)):
        r, blk, slot, hl = oracle.old_location(int(l[i]), int(h[i]), int(s[i]), int(t[i]), old_topo, L, H,
                                               old_tables)
        groups.setdefault((r, int(l[i]), int(kv[i])), []).append((i, blk, slot, hl))
    dims = np.arange(D, dtype=np.int64)
    for (r, ll, k), items in groups.items():
        idx = np.array([a[0] for a in items])
        blk, slot, hl = (np.array([a[j] for a in items], dtype=np.int64)[:, None] for j in (1, 2, 3))
        offs = element_offsets(layout, k, blk, slot, hl, dims[None, :], H_loc, bs, D, e) * e   # [n, D]
        vals = synthkv.bytes_at(offs.reshape(-1), e, w.seed, synthkv.SOURCE, r, ll, k)       # [n * D, e]
        out[idx] = vals.reshape(len(items), D * e)
    return out


def _gather(buf_u8: torch.Tensor, byte_offsets: np.ndarray, n: int) -> np.ndarray:
    idx = torch.from_numpy(byte_offsets[:, None] + np.arange(n, dtype=np.int64)).to(buf_u8.device)
    return buf_u8[idx].cpu().numpy()


def _check_staging(w, plan, inp, pair, buf, l0, l1, rng, nsamp=1500):
    L, H, D, e = w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes
    old_t, new_t = T(*w.old_topo), T(*w.new_topo)
    slices = oracle.pair_slices(old_t, new_t, L, H)
    ls, hs = slices[pair]
    ls = [x for x in ls if l0 <= x < l1]
    if not ls:
        return 0
    tok_off = oracle.token_offsets(inp.lens)
    _, offs = plan.query(*pair)
    s, t = _sample_tokens(rng, inp.lens, nsamp)
    n = len(s)
    l = np.array(ls)[rng.integers(0, len(ls), size=n)]
    l[: len(ls)] = ls[: n]                      # every layer of the window at least once
    kv = rng.integers(0, 2, size=n)
    h = np.array(hs)[rng.integers(0, len(hs), size=n)]
    at = np.array([oracle.staging_location(pair[0], pair[1], int(l[i]), int(kv[i]), int(h[i]), int(s[i]),
                                           int(t[i]), old_t, new_t, L, H, D, e, inp.lens, slices=slices,
                                           tok_off=tok_off) for i in range(n)], dtype=np.int64) - int(offs[l0])
    got = _gather(buf, at, D * e)
    want = _source_bytes(w, old_t, inp.old_tables, l, kv, h, s, t)
    bad = np.nonzero((got != want).any(axis=1))[0]
    assert bad.size == 0, f"staging {pair}: {bad.size} of {n} sampled rows differ (first: layer {l[bad[0]]}, " \
                          f"kv {kv[bad[0]]}, head {h[bad[0]]}, seq {s[bad[0]]}, token {t[bad[0]]})"
    return n


def _check_new_pool(w, inp, qn, dst, l0, l1, rng, nsamp=3000):
    L, H, D, e = w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes
    old_t, new_t = T(*w.old_topo), T(*w.new_topo)
    layers = [x for x in oracle.layers_of(qn, new_t, L) if l0 <= x < l1]
    heads = list(oracle.heads_of(qn, new_t, H))
    s, t = _sample_tokens(rng, inp.lens, nsamp)
    n = len(s)
    l = np.array(layers)[rng.integers(0, len(layers), size=n)]
    kv = rng.integers(0, 2, size=n)
    h = np.array(heads)[rng.integers(0, len(heads), size=n)]
    got = np.empty((n, D * e), np.uint8)
    for ll in set(l.tolist()):
        m = np.nonzero(l == ll)[0]
        loc = [oracle.new_location(ll, int(h[i]), int(s[i]), int(t[i]), new_t, L, H, inp.new_tables) for i in m]
        assert all(x[0] == qn for x in loc)
        store = dst.store[ll]
        ii = torch.tensor([[int(kv[i]), x[1], x[2], x[3]] for i, x in zip(m, loc)], device=store.device)
        rows = store[ii[:, 0], ii[:, 1], ii[:, 2], ii[:, 3]]          # [k, D]
        got[m] = rows.cpu().numpy().view(np.uint8).reshape(len(m), D * e)
    want = _source_bytes(w, old_t, inp.old_tables, l, kv, h, s, t)
    bad = np.nonzero((got != want).any(axis=1))[0]
    assert bad.size == 0, f"new pool: {bad.size} of {n} sampled rows differ"
    return n


def _check_new_pool_layout(w, inp, qn, dst, l0, l1, rng, layout, src_layout, nsamp=3000):
    """Sampled rows of a new pool the library writes in `layout`, read back through the layout's offsets;
    expected values come from the sources read in `src_layout`."""
    L, H, D, e = w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes
    old_t, new_t = T(*w.old_topo), T(*w.new_topo)
    H_loc = local_heads(H, new_t.tp)
    bs = inp.new_tables.block_size
    layers = [x for x in oracle.layers_of(qn, new_t, L) if l0 <= x < l1]
    heads = list(oracle.heads_of(qn, new_t, H))
    s, t = _sample_tokens(rng, inp.lens, nsamp)
    n = len(s)
    l = np.array(layers)[rng.integers(0, len(layers), size=n)]
    kv = rng.integers(0, 2, size=n)
    h = np.array(heads)[rng.integers(0, len(heads), size=n)]
    got = np.empty((n, D * e), np.uint8)
    dims = np.arange(D, dtype=np.int64)
    for ll in set(l.tolist()):
        for k in range(2):
            m = np.nonzero((l == ll) & (kv == k))[0]
            if m.size == 0:
                continue
            loc = [oracle.new_location(ll, int(h[i]), int(s[i]), int(t[i]), new_t, L, H, inp.new_tables) for i in m]
            assert all(x[0] == qn for x in loc)
            blk, slot, hl = (np.array([x[j] for x in loc], dtype=np.int64)[:, None] for j in (1, 2, 3))
            offs = element_offsets(layout, k, blk, slot, hl, dims[None, :], H_loc, bs, D, e) * e
            flat = dst.store[ll][k].reshape(-1).view(torch.uint8)
            byte_idx = torch.from_numpy((offs[:, :, None] + np.arange(e)).reshape(-1)).to(flat.device)
            got[m] = flat[byte_idx].cpu().numpy().reshape(m.size, D * e)
    want = _source_bytes(w, old_t, inp.old_tables, l, kv, h, s, t, layout=src_layout)
    bad = np.nonzero((got != want).any(axis=1))[0]
    assert bad.size == 0, f"new pool ({layout}): {bad.size} of {n} sampled rows differ"
    return n


def _live_mask(tables):
    m = np.zeros((tables.num_blocks, tables.block_size), dtype=bool)
    for s in range(tables.num_seqs):
        blk, slot = oracle.token_slots(tables, s)
        m[blk, slot] = True
    return m


def _check_live_rows_exactly(w, dst, qn, mask_dev):
    """Every byte of the new pool: differs from the sentinel exactly at live rows."""
    for l, store in dst.store.items():
        ref = torch.empty_like(store)
        for kv in range(2):
            synthkv.fill_sentinel_(ref[kv], w.seed, 0, qn, l, kv)
            changed = (ref[kv] != store[kv]).flatten(2).any(-1)          # [nb, bs]
            assert torch.equal(changed, mask_dev), f"layer {l} kv {kv}: written rows != live rows"
        del ref


def _check_sources_unchanged(w, src, r):
    for l, store in src.store.items():
        ref = torch.empty_like(store)
        for kv in range(2):
            synthkv.fill_pool_layer_(ref[kv], w.seed, r, l, kv)
        assert torch.equal(ref, store), f"source rank {r} layer {l} was modified"
        del ref


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", list(FULL))
def test_full_size_sampled(name):
    w = synthkv.WORKLOADS[name]
    inp = synthkv.make_inputs(w)
    L = w.num_layers
    ro, qn = w.role
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    W_old, W_new = plan.info.old_world, plan.info.new_world
    pairs_out = [(p.src, p.dst) for p in plan.pairs if p.src == ro]
    pairs_in = [(p.src, p.dst) for p in plan.pairs if p.dst == qn]
    pinfo = {(p.src, p.dst): p for p in plan.pairs}
    step = FULL[name] or L
    windows = [(a, min(L, a + step)) for a in range(0, L, step)]
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    ws = tio.workspace(plan, "cuda")
    stream = tio.current_stream()
    mask_dev = torch.from_numpy(_live_mask(inp.new_tables)).cuda()
    rng = np.random.default_rng(2024)
    checked = 0
    # windowed runs stream as a serving engine would: only the first pack and the first unpack expand
    # the block tables, every later call reuses their descriptors
    reuse = rk.REMP_KV_REUSE_DESCRIPTORS
    old_expanded = new_expanded = False
    for (l0, l1) in windows:
        log(f"[fullsize] {name} window [{l0}, {l1}) T={plan.info.total_tokens}")
        win = range(l0, l1)
        src = RankPool(w, w.old_topo, inp.old_tables, ro, "source", layers=win)
        dst = RankPool(w, w.new_topo, inp.new_tables, qn, "sentinel", layers=win)
        staging = tio.alloc_staging(plan, sorted(set(pairs_out) | set(pairs_in)), "cuda", window=(l0, l1))
        for (r, q) in pairs_in:
            p = pinfo[(r, q)]
            if r == ro or p.layer_end <= l0 or p.layer_begin >= l1:
                continue
            fp = RankPool(w, w.old_topo, inp.old_tables, r, "source", layers=win)
            extra = tio.alloc_staging(plan, [k for k in pinfo if k[0] == r and k != (r, q)], "cuda",
                                      window=(l0, l1))
            bufs = dict(extra)
            bufs[(r, q)] = staging[(r, q)]
            plan.pack(r, fp.arg, dto.dev, tio.staging_args(bufs, r, W_new, True), ws, ws.numel(), stream, l0, l1,
                      flags=reuse if old_expanded else 0)
            old_expanded = True
            torch.cuda.synchronize()
            assert tio.workspace_flag(ws) == 0
            del fp, extra, bufs
        plan.pack(ro, src.arg, dto.dev, tio.staging_args({k: staging[k] for k in pairs_out if k in staging},
                                                         ro, W_new, True), ws, ws.numel(), stream, l0, l1,
                  flags=reuse if old_expanded else 0)
        old_expanded = True
        torch.cuda.synchronize()
        assert tio.workspace_flag(ws) == 0
        plan.unpack(qn, tio.staging_args({k: staging[k] for k in pairs_in if k in staging}, qn, W_old, False),
                    dst.arg, dtn.host, dtn.dev, ws, ws.numel(), stream, l0, l1, flags=reuse if new_expanded else 0)
        new_expanded = True
        torch.cuda.synchronize()
        assert tio.workspace_flag(ws) == 0
        for pair in sorted(set(pairs_out) | set(pairs_in)):
            if pair in staging:
                checked += _check_staging(w, plan, inp, pair, staging[pair], l0, l1, rng)
        if dst.store:
            checked += _check_new_pool(w, inp, qn, dst, l0, l1, rng)
            _check_live_rows_exactly(w, dst, qn, mask_dev)
        _check_sources_unchanged(w, src, ro)
        log(f"[fullsize] {name} window [{l0}, {l1}) ok, {checked} sampled rows so far")
        del src, dst, staging
        torch.cuda.empty_cache()
    assert checked > 0


LAYOUT_FULL = [(1, 1, False), (2, 2, False), (0, 2, False), (2, 2, True), (1, 0, True)]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("lo,ln,local", LAYOUT_FULL)
def test_full_size_layouts(lo, ln, local):
    """The 70B GQA share at full size with HND / ROCm pools (staged, or with the local fast path):
    sampled staging and new-pool rows against the generator, sources untouched."""
    name = "gqa70b"
    w = synthkv.WORKLOADS[name]
    inp = synthkv.make_inputs(w)
    L = w.num_layers
    ro, qn = w.role
    plan = rk.Plan(w.old_topo, w.new_topo, shape_of(w), rk.HostTables.of(inp.old_tables))
    W_old, W_new = plan.info.old_world, plan.info.new_world
    skip = (lambda k: local and k[0] == k[1])
    pairs_out = [(p.src, p.dst) for p in plan.pairs if p.src == ro and not skip((p.src, p.dst))]
    pairs_in = [(p.src, p.dst) for p in plan.pairs if p.dst == qn and not skip((p.src, p.dst))]
    pinfo = {(p.src, p.dst): p for p in plan.pairs}
    windows = [(a, min(L, a + 20)) for a in range(0, L, 20)]
    dto, dtn = DeviceTables(inp.old_tables), DeviceTables(inp.new_tables)
    ws = tio.workspace(plan, "cuda")
    stream = tio.current_stream()
    fl = rk.REMP_KV_SKIP_LOCAL if local else 0
    rng = np.random.default_rng(77)
    checked = 0
    for (l0, l1) in windows:
        log(f"[fullsize layouts] old {lo} new {ln} local={local} window [{l0}, {l1})")
        win = range(l0, l1)
        src = RankPool(w, w.old_topo, inp.old_tables, ro, "source", layers=win, layout=lo)
        dst = RankPool(w, w.new_topo, inp.new_tables, qn, "sentinel", layers=win, layout=ln)
        staging = tio.alloc_staging(plan, sorted(set(pairs_out) | set(pairs_in)), "cuda", window=(l0, l1))
        for (r, q) in pairs_in:
            p = pinfo[(r, q)]
            if r == ro or p.layer_end <= l0 or p.layer_begin >= l1:
                continue
            fp = RankPool(w, w.old_topo, inp.old_tables, r, "source", layers=win, layout=lo)
            extra = tio.alloc_staging(plan, [k for k in pinfo if k[0] == r and k != (r, q) and not skip(k)], "cuda",
                                      window=(l0, l1))
            bufs = dict(extra)
            bufs[(r, q)] = staging[(r, q)]
            plan.pack(r, fp.arg, dto.dev, tio.staging_args(bufs, r, W_new, True), ws, ws.numel(), stream, l0, l1,
                      flags=fl)
            torch.cuda.synchronize()
            assert tio.workspace_flag(ws) == 0
            del fp, extra, bufs
        plan.pack(ro, src.arg, dto.dev, tio.staging_args({k: staging[k] for k in pairs_out if k in staging},
                                                         ro, W_new, True), ws, ws.numel(), stream, l0, l1, flags=fl)
        plan.unpack(qn, tio.staging_args({k: staging[k] for k in pairs_in if k in staging}, qn, W_old, False),
                    dst.arg, dtn.host, dtn.dev, ws, ws.numel(), stream, l0, l1, flags=fl)
        if local:
            plan.copy_local(ro, src.arg, dto.dev, dst.arg, dtn.host, dtn.dev, ws, ws.numel(), stream, l0, l1)
        torch.cuda.synchronize()
        assert tio.workspace_flag(ws) == 0
        for pair in sorted(set(pairs_out) | set(pairs_in)):
            if pair in staging:
                checked += _check_staging_layout(w, plan, inp, pair, staging[pair], l0, l1, rng, lo)
        if dst.store:
            checked += _check_new_pool_layout(w, inp, qn, dst, l0, l1, rng, ln, lo)
        _check_sources_unchanged(w, src, ro)
        del src, dst, staging
        torch.cuda.empty_cache()
    assert checked > 0


def _check_staging_layout(w, plan, inp, pair, buf, l0, l1, rng, lo, nsamp=1500):
    """Sampled staging rows of a pair when the sources are read in layout `lo`."""
    L, H, D, e = w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes
    old_t, new_t = T(*w.old_topo), T(*w.new_topo)
    slices = oracle.pair_slices(old_t, new_t, L, H)
    ls, hs = slices[pair]
    ls = [x for x in ls if l0 <= x < l1]
    if not ls:
        return 0
    tok_off = oracle.token_offsets(inp.lens)
    _, offs = plan.query(*pair)
    s, t = _sample_tokens(rng, inp.lens, nsamp)
    n = len(s)
    l = np.array(ls)[rng.integers(0, len(ls), size=n)]
    l[: len(ls)] = ls[: n]
    kv = rng.integers(0, 2, size=n)
    h = np.array(hs)[rng.integers(0, len(hs), size=n)]
    at = np.array([oracle.staging_location(pair[0], pair[1], int(l[i]), int(kv[i]), int(h[i]), int(s[i]),
                                           int(t[i]), old_t, new_t, L, H, D, e, inp.lens, slices=slices,
                                           tok_off=tok_off) for i in range(n)], dtype=np.int64) - int(offs[l0])
    got = _gather(buf, at, D * e)
    want = _source_bytes(w, old_t, inp.old_tables, l, kv, h, s, t, layout=lo)
    bad = np.nonzero((got != want).any(axis=1))[0]
    assert bad.size == 0, f"staging {pair} ({lo}): {bad.size} of {n} sampled rows differ"
    return n
