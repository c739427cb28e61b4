"""Pins of the weight-shard oracle (Section 3.3) against things other than itself.

* two hand-derived worked examples (tests/golden/weights_hand_*.json);
* a second, element-by-element formulation (tests/bruteforce_weights.py) on
  tiny decoders over many topologies, uneven pipeline partitions and
  replicated KV heads included;
* the mathematics of tensor parallelism: with float64 weights, a decoder
  layer computed shard by shard (grouped-query attention on each rank's local
  heads, row-parallel partial sums, vocabulary-parallel embedding lookups)
  equals the same layer computed with the full weights;
* planted mistakes in the oracle, each of which one of the above catches.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synthkv
from oracle import weights as ow
from oracle.migration import Topology

import bruteforce_weights as bw
from weights_harness import load_golden, oracle_tensors

GOLDENS = ["weights_hand_tp2pp2.json", "weights_hand_tp4_gqa.json"]


def _check_golden(name):
    g, names, tensors, _ = load_golden(name)
    tp, pp = g["topo"]
    topo = Topology(tp, pp)
    for rank in range(tp * pp):
        got = ow.rank_shards(tensors, topo, g["num_layers"], rank)
        want = g["expected"].get(str(rank), {})
        assert sorted(names[i] for i in got) == sorted(want), (name, rank)
        for i, arr in got.items():
            np.testing.assert_array_equal(arr, np.array(want[names[i]], dtype=np.uint16), err_msg=f"{name} {rank}")


@pytest.mark.parametrize("name", GOLDENS)
def test_golden_hand_example(name):
    _check_golden(name)


# ---------------------------------------------------------------------------
# brute force
# ---------------------------------------------------------------------------

TOPOS = {
    "tiny": [(1, 1), (2, 1), (4, 1), (8, 1), (1, 2), (2, 2), (4, 2), (8, 2), (2, 4), (1, 4),
             (2, 2, (0, 1, 4)), (4, 3, (0, 2, 3, 4)), (8, 2, (0, 3, 4))],
    "odd": [(1, 1), (3, 1), (6, 1), (1, 3), (3, 3), (6, 3), (3, 2, (0, 2, 3)), (6, 2, (0, 1, 3))],
}


def _brute_case(spec, topo_t):
    tp, pp = topo_t[0], topo_t[1]
    starts = topo_t[2] if len(topo_t) > 2 else None
    store = synthkv.models.host_store(spec)
    tensors = oracle_tensors(spec, store)
    topo = Topology(tp, pp, starts)
    for rank in range(tp * pp):
        got = ow.rank_shards(tensors, topo, spec.num_layers, rank)
        want = bw.shards(tensors, tp, pp, spec.num_layers, rank, starts)
        assert sorted(got) == sorted(want), (topo_t, rank)
        for i in got:
            np.testing.assert_array_equal(got[i], np.array(want[i], dtype=got[i].dtype),
                                          err_msg=f"{spec.name} {topo_t} rank {rank} tensor {i}")


@pytest.mark.parametrize("spec_name,topo", [(s, t) for s, ts in TOPOS.items() for t in ts])
def test_bruteforce_agrees(spec_name, topo):
    _brute_case(synthkv.DECODERS[spec_name], topo)


def test_every_part_byte_reaches_some_rank():
    """Coverage: over all ranks of a topology, every element of every part is in some shard
    (checked by value: parts hold distinct hash words with overwhelming probability)."""
    spec = synthkv.TINY_DECODER
    store = synthkv.models.host_store(spec)
    tensors = oracle_tensors(spec, store)
    for tp, pp in [(2, 2), (8, 1), (4, 4)]:
        topo = Topology(tp, pp)
        seen = set()
        for r in range(tp * pp):
            for arr in ow.rank_shards(tensors, topo, spec.num_layers, r).values():
                seen.update(np.unique(arr).tolist())
        for _, parts in tensors:
            for a, _, _ in parts:
                assert set(np.unique(a).tolist()) <= seen


# ---------------------------------------------------------------------------
# the mathematics of tensor parallelism, in float64
# ---------------------------------------------------------------------------

def _float_decoder(spec, rng):
    """Float64 weights in the oracle's tensor form (same inventory and splits as the spec)."""
    tensors = []
    for t in spec.tensors():
        parts = [(rng.standard_normal((p.rows, p.cols)), p.split, p.units) for p in t.parts]
        tensors.append((t.layer, parts))
    return tensors


def _silu(z):
    return z / (1.0 + np.exp(-z))


def _attention(q, k, v, heads, kv_heads, D):
    """Causal grouped-query attention: query head h reads KV head h // (heads / kv_heads)."""
    T = q.shape[0]
    q = q.reshape(T, heads, D)
    k = k.reshape(T, kv_heads, D)
    v = v.reshape(T, kv_heads, D)
    group = heads // kv_heads
    mask = np.triu(np.full((T, T), -np.inf), 1)
    out = np.empty((T, heads, D))
    for h in range(heads):
        s = q[:, h] @ k[:, h // group].T / np.sqrt(D) + mask
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        out[:, h] = p @ v[:, h // group]
    return out.reshape(T, heads * D)


def _layer_full(tensors, l_index, x, spec):
    """One decoder layer (without norms' arithmetic) and the embedding / LM head, full weights."""
    emb, n_in, qkv, o, n_post, gu, down = (tensors[0],) + tuple(tensors[1 + 6 * l_index + j] for j in range(6))
    Wq, Wk, Wv = (qkv[1][j][0] for j in range(3))
    Wo = o[1][0][0]
    Wg, Wu = gu[1][0][0], gu[1][1][0]
    Wd = down[1][0][0]
    attn = _attention(x @ Wq.T, x @ Wk.T, x @ Wv.T, spec.heads, spec.kv_heads, spec.head_dim)
    h1 = attn @ Wo.T
    h2 = (_silu(x @ Wg.T) * (x @ Wu.T)) @ Wd.T
    return h1, h2, n_in[1][0][0], n_post[1][0][0]


def _layer_sharded(tensors, l_index, x, spec, tp):
    """The same layer computed rank by rank from the oracle's shards, then combined."""
    H, Hkv, D, I = spec.heads, spec.kv_heads, spec.head_dim, spec.intermediate
    topo = Topology(tp, 1)
    L = spec.num_layers
    qkv_i, o_i, gu_i, down_i = 2 + 6 * l_index, 3 + 6 * l_index, 5 + 6 * l_index, 6 + 6 * l_index
    n_in_i, n_post_i = 1 + 6 * l_index, 4 + 6 * l_index
    h_loc = H // tp
    kv_loc = Hkv // tp if tp <= Hkv else 1
    h1 = np.zeros((x.shape[0], spec.hidden))
    h2 = np.zeros((x.shape[0], spec.hidden))
    norms = []
    for t in range(tp):
        s = ow.rank_shards(tensors, topo, L, t)
        y = x @ s[qkv_i].T
        q, k, v = y[:, :h_loc * D], y[:, h_loc * D:(h_loc + kv_loc) * D], y[:, (h_loc + kv_loc) * D:]
        assert v.shape[1] == kv_loc * D
        attn_t = _attention(q, k, v, h_loc, kv_loc, D)
        h1 += attn_t @ s[o_i].T                       # row-parallel: partial sums
        gu = x @ s[gu_i].T
        i_loc = I // tp
        h2 += (_silu(gu[:, :i_loc]) * gu[:, i_loc:]) @ s[down_i].T
        norms.append((s[n_in_i], s[n_post_i]))
    return h1, h2, norms


@pytest.mark.parametrize("tp", [1, 2, 4, 8])
def test_sharded_layer_equals_full_layer(tp):
    spec = synthkv.TINY_DECODER
    _check_tp_math(spec, tp)


@pytest.mark.parametrize("tp", [3, 6])
def test_sharded_layer_equals_full_layer_odd(tp):
    _check_tp_math(synthkv.ODD_DECODER, tp)


def _check_tp_math(spec, tp):
    rng = np.random.default_rng(100 + tp)
    tensors = _float_decoder(spec, rng)
    T = 5
    x = rng.standard_normal((T, spec.hidden))
    for l_index in range(spec.num_layers):
        f1, f2, n_in, n_post = _layer_full(tensors, l_index, x, spec)
        s1, s2, norms = _layer_sharded(tensors, l_index, x, spec, tp)
        np.testing.assert_allclose(s1, f1, rtol=1e-9, atol=1e-9)
        np.testing.assert_allclose(s2, f2, rtol=1e-9, atol=1e-9)
        for a, b in norms:
            np.testing.assert_array_equal(a, n_in)
            np.testing.assert_array_equal(b, n_post)
    # vocabulary-parallel embedding (masked lookups summed) and LM head (logits concatenated)
    V = spec.vocab
    topo = Topology(tp, 1)
    E = tensors[0][1][0][0]
    W = tensors[-1][1][0][0]
    ids = rng.integers(0, V, size=17)
    emb = np.zeros((ids.size, spec.hidden))
    logits = []
    hdn = rng.standard_normal((3, spec.hidden))
    for t in range(tp):
        s = ow.rank_shards(tensors, topo, spec.num_layers, t)
        lo = t * (V // tp)
        mine = (ids >= lo) & (ids < lo + V // tp)
        emb[mine] += s[0][ids[mine] - lo]
        logits.append(hdn @ s[len(tensors) - 1].T)
    np.testing.assert_array_equal(emb, E[ids])
    np.testing.assert_allclose(np.concatenate(logits, axis=1), hdn @ W.T, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# planted mistakes: each one must be caught by a pin above
# ---------------------------------------------------------------------------

def _pins_pass():
    try:
        for g in GOLDENS:
            _check_golden(g)
        _check_tp_math(synthkv.TINY_DECODER, 4)
        _check_tp_math(synthkv.TINY_DECODER, 8)
        _check_tp_math(synthkv.ODD_DECODER, 6)
        _brute_case(synthkv.TINY_DECODER, (2, 2, (0, 1, 4)))
    except (AssertionError, ValueError, IndexError):
        return False
    return True


def _mutant_replica_by_modulo(t, tp, units):
    if tp <= units:
        per = units // tp
        return range(t * per, (t + 1) * per)
    return range(t % units, t % units + 1)


def _mutant_units_shifted(t, tp, units):
    if tp <= units:
        per = units // tp
        a = (t * per + 1) % units
        return range(a, a + per) if a + per <= units else range(0, per)
    u = t // (tp // units)
    return range(u, u + 1)


def _mutant_cols_as_rows(a, split, units, t, tp):
    return _orig_part_slice(a, ow.SPLIT_ROWS if split == ow.SPLIT_COLS else split, units, t, tp)


def _mutant_first_last_swapped(stage, layer, topo, L):
    if layer == ow.FIRST_STAGE:
        return stage == topo.pp - 1
    if layer == ow.LAST_STAGE:
        return stage == 0
    return oracle.pp_owner(layer, topo, L) == stage


def _mutant_parts_reversed(parts, t, tp):
    return np.concatenate([ow.part_slice(a, s, u, t, tp) for (a, s, u) in reversed(list(parts))], axis=0)


def _mutant_even_layers(stage, layer, topo, L):
    if layer < 0:
        return _orig_stage_holds(stage, layer, topo, L)
    return layer // (L // topo.pp if L >= topo.pp else 1) == stage


_orig_part_slice = ow.part_slice
_orig_stage_holds = ow.stage_holds

MUTANTS = {
    "replica_by_modulo": ("units_kept", _mutant_replica_by_modulo),
    "units_shifted": ("units_kept", _mutant_units_shifted),
    "cols_as_rows": ("part_slice", _mutant_cols_as_rows),
    "first_last_swapped": ("stage_holds", _mutant_first_last_swapped),
    "parts_reversed": ("shard", _mutant_parts_reversed),
    "ignores_partition": ("stage_holds", _mutant_even_layers),
}


def test_pins_pass_unmodified():
    assert _pins_pass()


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    attr, fn = MUTANTS[mutant]
    monkeypatch.setattr(ow, attr, fn)
    assert not _pins_pass(), f"planted mistake {mutant} passed every pin"
