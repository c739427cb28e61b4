"""Synthetic decoder models for the weight-shard rebuild: tensor inventories and seeded store contents.

A model here is only a list of parameter tensors with their shapes and the
tensor-parallel split each one takes (the usual Megatron-style split of a
Llama-architecture decoder, as vLLM lays it out on the GPU):

    embed_tokens        [V, hidden]      rows split by vocabulary entry     first stage
    per layer:
      input_layernorm   [1, hidden]      replicated
      qkv_proj          q_proj [Hq*D, hidden] | k_proj [Hkv*D, hidden] | v_proj [Hkv*D, hidden],
                        each split by heads along rows (K and V replicated when TP > Hkv)
      o_proj            [hidden, Hq*D]   columns split by heads
      post_attention_layernorm [1, hidden] replicated
      gate_up_proj      gate_proj [I, hidden] | up_proj [I, hidden], rows split
      down_proj         [hidden, I]      columns split
    norm                [1, hidden]      replicated                         last stage
    lm_head             [V, hidden]      rows split by vocabulary entry     last stage

Variants: Q/K/V biases (Qwen2, as in DeepSeek-R1-Distill-Qwen-32B) split by
heads like their weights; per-head Q/K norm weights (Qwen3), replicated; a
mixture-of-experts MLP (Qwen3-30B-A3B) whose experts are each split by TP
like a dense MLP, with a replicated router.

The store holds every part ("q_proj", "k_proj" ...) whole, as the
checkpoint does; GPU tensors stack the rank's slices of their parts.  Shapes
follow the models of the paper's evaluation (Llama2-7B, Llama3-70B,
DeepSeek-R1-Distill-Qwen-32B, Qwen3-30B-A3B); contents are seeded hash words,
values are never interpreted.  Nothing here slices.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Tuple

import numpy as np
import torch

from .gen import fill_words_

REPLICATED, SPLIT_ROWS, SPLIT_COLS = 0, 1, 2
FIRST_STAGE, LAST_STAGE = -1, -2
WEIGHTS = 0x5745   # stream tag of store contents


@dataclass(frozen=True)
class StorePart:
    name: str
    rows: int
    cols: int
    split: int
    units: int
    key: int          # generator stream of its contents


@dataclass(frozen=True)
class GpuTensor:
    name: str
    layer: int                     # >= 0, FIRST_STAGE or LAST_STAGE
    parts: Tuple[StorePart, ...]   # stacked along rows in the shard


@dataclass(frozen=True)
class DecoderSpec:
    name: str
    num_layers: int
    hidden: int
    heads: int
    kv_heads: int
    head_dim: int
    intermediate: int
    vocab: int
    elem_bytes: int
    seed: int
    qkv_bias: bool = False        # Qwen2-style biases on Q, K, V
    qk_norm: bool = False         # Qwen3-style per-head RMSNorm weights on Q and K
    num_experts: int = 0          # > 0: a mixture-of-experts MLP of that many experts
    moe_intermediate: int = 0     # intermediate size of one expert

    def tensors(self, layers=None) -> List[GpuTensor]:
        """GPU tensors in load order: embedding, then each layer's, then final norm and LM head.
        `layers` restricts the decoder layers listed (the embedding / head are always listed)."""
        H, Hkv, D, h, I, V = self.heads, self.kv_heads, self.head_dim, self.hidden, self.intermediate, self.vocab
        E, Ie = self.num_experts, self.moe_intermediate

        def part(name, rows, cols, split, units, key):
            return StorePart(name, rows, cols, split, units, key)

        out = [GpuTensor("embed_tokens", FIRST_STAGE, (part("embed_tokens", V, h, SPLIT_ROWS, V, 1),))]
        for l in range(self.num_layers):
            if layers is not None and l not in layers:
                continue
            k0 = (l + 1) << 12      # generator streams of layer l's parts: k0 + part number
            p = f"layers.{l}."
            t = [GpuTensor(p + "input_layernorm", l, (part(p + "input_layernorm", 1, h, REPLICATED, 1, k0),)),
                 GpuTensor(p + "qkv_proj", l,
                           (part(p + "q_proj", H * D, h, SPLIT_ROWS, H, k0 + 1),
                            part(p + "k_proj", Hkv * D, h, SPLIT_ROWS, Hkv, k0 + 2),
                            part(p + "v_proj", Hkv * D, h, SPLIT_ROWS, Hkv, k0 + 3)))]
            if self.qkv_bias:   # biases as column vectors: they stack like the weights' rows
                t.append(GpuTensor(p + "qkv_bias", l,
                                   (part(p + "q_bias", H * D, 1, SPLIT_ROWS, H, k0 + 4),
                                    part(p + "k_bias", Hkv * D, 1, SPLIT_ROWS, Hkv, k0 + 5),
                                    part(p + "v_bias", Hkv * D, 1, SPLIT_ROWS, Hkv, k0 + 6))))
            if self.qk_norm:
                t.append(GpuTensor(p + "q_norm", l, (part(p + "q_norm", 1, D, REPLICATED, 1, k0 + 7),)))
                t.append(GpuTensor(p + "k_norm", l, (part(p + "k_norm", 1, D, REPLICATED, 1, k0 + 8),)))
            t.append(GpuTensor(p + "o_proj", l, (part(p + "o_proj", h, H * D, SPLIT_COLS, H, k0 + 9),)))
            t.append(GpuTensor(p + "post_attention_layernorm", l,
                               (part(p + "post_attention_layernorm", 1, h, REPLICATED, 1, k0 + 10),)))
            if E:
                # experts under tensor parallelism: every expert's gate / up rows and down columns split by TP;
                # the router is replicated.  Fused as [expert][gate | up][rows][hidden] and [expert][hidden][cols].
                t.append(GpuTensor(p + "router", l, (part(p + "router", E, h, REPLICATED, 1, k0 + 11),)))
                w13 = []
                for e in range(E):
                    w13.append(part(p + f"experts.{e}.gate_proj", Ie, h, SPLIT_ROWS, Ie, k0 + 16 + 3 * e))
                    w13.append(part(p + f"experts.{e}.up_proj", Ie, h, SPLIT_ROWS, Ie, k0 + 17 + 3 * e))
                t.append(GpuTensor(p + "experts.w13", l, tuple(w13)))
                t.append(GpuTensor(p + "experts.w2", l,
                                   tuple(part(p + f"experts.{e}.down_proj", h, Ie, SPLIT_COLS, Ie, k0 + 18 + 3 * e)
                                         for e in range(E))))
            else:
                t.append(GpuTensor(p + "gate_up_proj", l,
                                   (part(p + "gate_proj", I, h, SPLIT_ROWS, I, k0 + 12),
                                    part(p + "up_proj", I, h, SPLIT_ROWS, I, k0 + 13))))
                t.append(GpuTensor(p + "down_proj", l, (part(p + "down_proj", h, I, SPLIT_COLS, I, k0 + 14),)))
            out += t
        out += [GpuTensor("norm", LAST_STAGE, (part("norm", 1, h, REPLICATED, 1, 2),)),
                GpuTensor("lm_head", LAST_STAGE, (part("lm_head", V, h, SPLIT_ROWS, V, 3),))]
        return out

    def store_parts(self, layers=None) -> List[StorePart]:
        return [p for t in self.tensors(layers) for p in t.parts]

    @property
    def numpy_dtype(self):
        return {1: np.uint8, 2: np.uint16, 4: np.uint32}[self.elem_bytes]


TINY_DECODER = DecoderSpec("tiny", num_layers=4, hidden=64, heads=8, kv_heads=2, head_dim=8, intermediate=96,
                           vocab=128, elem_bytes=2, seed=11)
# row lengths that are not multiples of 16 bytes: copies fall back to narrower vectors
ODD_DECODER = DecoderSpec("odd", num_layers=3, hidden=36, heads=6, kv_heads=3, head_dim=6, intermediate=30,
                          vocab=42, elem_bytes=2, seed=12)
TINY_BIAS = DecoderSpec("tiny-bias", num_layers=2, hidden=32, heads=4, kv_heads=2, head_dim=8, intermediate=48,
                        vocab=64, elem_bytes=2, seed=15, qkv_bias=True)
TINY_MOE = DecoderSpec("tiny-moe", num_layers=2, hidden=32, heads=8, kv_heads=2, head_dim=4, intermediate=0,
                       vocab=64, elem_bytes=2, seed=16, qk_norm=True, num_experts=4, moe_intermediate=16)
LLAMA2_7B = DecoderSpec("llama2-7b", num_layers=32, hidden=4096, heads=32, kv_heads=32, head_dim=128,
                        intermediate=11008, vocab=32000, elem_bytes=2, seed=13)
LLAMA3_70B = DecoderSpec("llama3-70b", num_layers=80, hidden=8192, heads=64, kv_heads=8, head_dim=128,
                         intermediate=28672, vocab=128256, elem_bytes=2, seed=14)
# DeepSeek-R1-Distill-Qwen-32B (Qwen2 architecture: biases on Q, K, V)
QWEN2_32B = DecoderSpec("deepseek-r1-distill-qwen-32b", num_layers=64, hidden=5120, heads=40, kv_heads=8,
                        head_dim=128, intermediate=27648, vocab=152064, elem_bytes=2, seed=17, qkv_bias=True)
# Qwen3-30B-A3B (mixture of 128 experts, per-head Q/K norms)
QWEN3_30B_A3B = DecoderSpec("qwen3-30b-a3b", num_layers=48, hidden=2048, heads=32, kv_heads=4, head_dim=128,
                            intermediate=0, vocab=151936, elem_bytes=2, seed=18, qk_norm=True, num_experts=128,
                            moe_intermediate=768)
DECODERS = {d.name: d for d in (TINY_DECODER, ODD_DECODER, TINY_BIAS, TINY_MOE, LLAMA2_7B, LLAMA3_70B, QWEN2_32B,
                                QWEN3_30B_A3B)}


def part_nbytes(spec: DecoderSpec, p: StorePart) -> int:
    return p.rows * p.cols * spec.elem_bytes


def fill_part_(buf: torch.Tensor, spec: DecoderSpec, p: StorePart) -> torch.Tensor:
    """Fill the flat uint8 tensor `buf` (length >= the part's bytes rounded up to 4) with the part's contents."""
    n = (part_nbytes(spec, p) + 3) // 4 * 4
    return fill_words_(buf[:n], spec.seed, WEIGHTS, p.key)


def host_store(spec: DecoderSpec, layers=None, pin: bool = False, fill_device=None,
               chunk_bytes: int = 256 << 20, tensors=None) -> Dict[str, torch.Tensor]:
    """{part name: flat uint8 host tensor} holding every store part whole
    (of `tensors` if given, else of every tensor of `layers`).

    pin=True allocates page-locked memory (one allocation per part).  With
    fill_device (e.g. "cuda") contents are generated there, chunk by chunk, and
    copied to the host: the same bytes, much faster than on the CPU.
    """
    out = {}
    parts = spec.store_parts(layers) if tensors is None else [p for t in tensors for p in t.parts]
    for p in parts:
        n = part_nbytes(spec, p)
        padded = (n + 3) // 4 * 4
        t = torch.empty(padded, dtype=torch.uint8, pin_memory=pin)
        if fill_device is None:
            fill_part_(t, spec, p)
        else:
            _fill_via_device(t, spec, p, fill_device, chunk_bytes)
        out[p.name] = t
    return out


def _fill_via_device(t: torch.Tensor, spec: DecoderSpec, p: StorePart, device, chunk_bytes: int) -> None:
    # word i of the part is hash(i ^ key): generate word ranges on the device and copy them over
    from .gen import hash_words, stream_key
    key = stream_key(spec.seed, WEIGHTS, p.key)
    words = t.view(torch.int32)
    n = words.numel()
    step = chunk_bytes // 4
    for a in range(0, n, step):
        b = min(n, a + step)
        idx = torch.arange(a, b, dtype=torch.int64, device=device)
        words[a:b].copy_(hash_words(idx, key))
    if str(device).startswith("cuda"):
        torch.cuda.synchronize()


def part_array(spec: DecoderSpec, store: Dict[str, torch.Tensor], p: StorePart) -> np.ndarray:
    """[rows][cols] numpy view of a store part."""
    n = part_nbytes(spec, p)
    return store[p.name][:n].numpy().view(spec.numpy_dtype).reshape(p.rows, p.cols)
