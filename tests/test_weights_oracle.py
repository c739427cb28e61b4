"""Pins of the weight-shard oracle (Section 3.3) against things other than itself.

* two hand-derived worked examples (tests/golden/weights_hand_*.json);
* a second, element-by-element formulation (tests/bruteforce_weights.py) on
  tiny decoders over many topologies, uneven pipeline partitions and
  replicated KV heads included;
* the mathematics of tensor parallelism: with float64 weights, a decoder
  layer computed shard by shard (grouped-query attention on each rank's local
  heads with Q/K/V biases and per-head Q/K norms where the model has them,
  row-parallel partial sums, every expert of a mixture of experts,
  vocabulary-parallel embedding lookups) equals the same layer computed with
  the full weights;
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
    "tiny-bias": [(1, 1), (2, 2), (4, 1), (8, 1)],
    "tiny-moe": [(1, 1), (2, 2), (4, 1), (8, 2)],
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


def _rms(z, w):
    return z / np.sqrt((z * z).mean(axis=-1, keepdims=True) + 1e-6) * w


def _attn_in(y, nq, nkv, D, qn=None, kn=None):
    """Split a fused Q|K|V projection output; apply per-head Q/K norms when given."""
    T = y.shape[0]
    q, k, v = y[:, :nq * D], y[:, nq * D:(nq + nkv) * D], y[:, (nq + nkv) * D:]
    assert v.shape[1] == nkv * D
    if qn is not None:
        q = _rms(q.reshape(T, nq, D), qn.reshape(-1)).reshape(T, nq * D)
        k = _rms(k.reshape(T, nkv, D), kn.reshape(-1)).reshape(T, nkv * D)
    return q, k, v


def _layer(get, x, spec, l, tp):
    """Attention and MLP outputs of layer l, from the GPU tensors `get(name)` of one tensor rank
    (tp = 1: the full weights).  Row-parallel outputs are partial sums over ranks."""
    H, Hkv, D = spec.heads, spec.kv_heads, spec.head_dim
    h_loc = H // tp
    kv_loc = Hkv // tp if tp <= Hkv else 1
    p = f"layers.{l}."
    y = x @ get(p + "qkv_proj").T
    if spec.qkv_bias:
        y = y + get(p + "qkv_bias").reshape(-1)
    qn = get(p + "q_norm") if spec.qk_norm else None
    kn = get(p + "k_norm") if spec.qk_norm else None
    q, k, v = _attn_in(y, h_loc, kv_loc, D, qn, kn)
    attn = _attention(q, k, v, h_loc, kv_loc, D) @ get(p + "o_proj").T
    if spec.num_experts:
        E, h = spec.num_experts, spec.hidden
        i_loc = spec.moe_intermediate // tp
        logits = x @ get(p + "router").T
        g = np.exp(logits - logits.max(axis=1, keepdims=True))
        g /= g.sum(axis=1, keepdims=True)            # every expert weighted (a dense mixture checks them all)
        w13, w2 = get(p + "experts.w13"), get(p + "experts.w2")
        mlp = np.zeros((x.shape[0], h))
        for e in range(E):
            gu = x @ w13[e * 2 * i_loc:(e + 1) * 2 * i_loc].T
            mlp += g[:, e:e + 1] * ((_silu(gu[:, :i_loc]) * gu[:, i_loc:]) @ w2[e * h:(e + 1) * h].T)
    else:
        i_loc = spec.intermediate // tp
        gu = x @ get(p + "gate_up_proj").T
        mlp = (_silu(gu[:, :i_loc]) * gu[:, i_loc:]) @ get(p + "down_proj").T
    return attn, mlp


@pytest.mark.parametrize("tp", [1, 2, 4, 8])
def test_sharded_layer_equals_full_layer(tp):
    _check_tp_math(synthkv.TINY_DECODER, tp)


@pytest.mark.parametrize("tp", [3, 6])
def test_sharded_layer_equals_full_layer_odd(tp):
    _check_tp_math(synthkv.ODD_DECODER, tp)


@pytest.mark.parametrize("spec_name,tp", [("tiny-bias", 2), ("tiny-bias", 4), ("tiny-moe", 2), ("tiny-moe", 4),
                                          ("tiny-moe", 8)])
def test_sharded_layer_equals_full_layer_variants(spec_name, tp):
    """Q/K/V biases (Qwen2), per-head Q/K norms and a mixture of experts (Qwen3 MoE)."""
    _check_tp_math(synthkv.DECODERS[spec_name], tp)


def _check_tp_math(spec, tp):
    rng = np.random.default_rng(100 + tp)
    tensors = _float_decoder(spec, rng)
    names = [t.name for t in spec.tensors()]
    index = {n: i for i, n in enumerate(names)}
    # the full-weight GPU tensor: its parts, whole, stacked along rows
    full = {n: np.concatenate([a for (a, _, _) in tensors[i][1]], axis=0) for n, i in index.items()}
    topo = Topology(tp, 1)
    L = spec.num_layers
    shards = [ow.rank_shards(tensors, topo, L, t) for t in range(tp)]
    T = 5
    x = rng.standard_normal((T, spec.hidden))
    for l in range(L):
        f_attn, f_mlp = _layer(lambda n: full[n], x, spec, l, 1)
        s_attn = np.zeros_like(f_attn)
        s_mlp = np.zeros_like(f_mlp)
        for t in range(tp):
            a, m = _layer(lambda n: shards[t][index[n]], x, spec, l, tp)
            s_attn += a
            s_mlp += m
        np.testing.assert_allclose(s_attn, f_attn, rtol=1e-9, atol=1e-9)
        np.testing.assert_allclose(s_mlp, f_mlp, rtol=1e-9, atol=1e-9)
        for n in ("input_layernorm", "post_attention_layernorm", "q_norm", "k_norm", "router"):
            if f"layers.{l}.{n}" in index:
                for t in range(tp):
                    np.testing.assert_array_equal(shards[t][index[f"layers.{l}.{n}"]], full[f"layers.{l}.{n}"])
    # vocabulary-parallel embedding (masked lookups summed) and LM head (logits concatenated)
    V = spec.vocab
    E, W = full["embed_tokens"], full["lm_head"]
    ids = rng.integers(0, V, size=17)
    emb = np.zeros((ids.size, spec.hidden))
    logits = []
    hdn = rng.standard_normal((3, spec.hidden))
    for t in range(tp):
        lo = t * (V // tp)
        mine = (ids >= lo) & (ids < lo + V // tp)
        emb[mine] += shards[t][index["embed_tokens"]][ids[mine] - lo]
        logits.append(hdn @ shards[t][index["lm_head"]].T)
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
