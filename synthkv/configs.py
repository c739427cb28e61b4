"""The five synthetic KV-migration workloads.

Each workload fixes a model's KV shape, a population of live sequences, the
block-table construction for the old and the new paged pool, and a topology
switch (old TP/PP -> new TP/PP).  Nothing here computes ownership or moves
data; it only describes inputs.

The shapes follow the models of the paper's evaluation table (Llama2-7B:
32 layers x 32 KV heads; Llama3-70B: 80 layers x 8 KV heads; Qwen3-30B-A3B:
48 layers x 4 KV heads; DeepSeek-R1-Distill-Qwen-32B: 64 layers x 8 KV heads;
head_dim 128).
The 40 x 40 "13B-shaped" workload is a synthetic MHA shape that is not one of
the paper's models.  The paper does not describe the KV population at switch
time, so sequence-length laws are synthetic stand-ins: uniform for the small
MHA cases, lognormal (sigma 0.5, around the stated median) for the serving
cases, and fixed 128k-token sequences for the long-context case.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Tuple


@dataclass(frozen=True)
class KVWorkload:
    name: str
    num_layers: int
    num_kv_heads: int
    head_dim: int
    elem_bytes: int
    dtype: str                      # "fp16" | "bf16" | "fp8" ... (bits are copied, never interpreted)
    old_block_size: int
    new_block_size: int
    num_seqs: int
    # ("uniform", lo, hi) | ("lognormal", median, sigma, cap) | ("fixed", n)
    length_law: Tuple
    # ("fixed", num_blocks) | ("slack", factor) | ("fragmented", occupied_fraction)
    pool_law: Tuple
    old_topo: Tuple[int, int]       # (tp, pp)
    new_topo: Tuple[int, int]
    # "all": every old rank packs and every new rank unpacks on one GPU;
    # (old_rank, new_rank): the GPU plays one old rank and one new rank.
    role: object
    seed: int
    description: str = ""

    def replace(self, **kw) -> "KVWorkload":
        return dataclasses.replace(self, **kw)

    @property
    def old_world(self) -> int:
        return self.old_topo[0] * self.old_topo[1]

    @property
    def new_world(self) -> int:
        return self.new_topo[0] * self.new_topo[1]


TINY = KVWorkload(
    name="tiny",
    num_layers=4, num_kv_heads=8, head_dim=64, elem_bytes=2, dtype="fp16",
    old_block_size=16, new_block_size=16,
    num_seqs=4, length_law=("uniform", 1, 256),
    pool_law=("fixed", 128),
    old_topo=(2, 1), new_topo=(1, 2), role="all", seed=0,
    description="L4 H8 D64 fp16 bs16, 4 seqs U[1,256], 128-block pools, TP2/PP1 -> TP1/PP2, all ranks",
)

MHA_7B = KVWorkload(
    name="mha7b",
    num_layers=32, num_kv_heads=32, head_dim=128, elem_bytes=2, dtype="bf16",
    old_block_size=16, new_block_size=16,
    num_seqs=64, length_law=("uniform", 512, 4096),
    pool_law=("slack", 1.1),
    old_topo=(4, 1), new_topo=(2, 2), role=(0, 0), seed=1,
    description="L32 H32 D128 bf16 bs16, 64 seqs U[512,4096], TP4/PP1 -> TP2/PP2, old rank 0 / new rank 0",
)

MHA_13B = KVWorkload(
    name="mha13b",
    num_layers=40, num_kv_heads=40, head_dim=128, elem_bytes=2, dtype="bf16",
    old_block_size=16, new_block_size=16,
    num_seqs=128, length_law=("lognormal", 1500, 0.5, 8192),
    pool_law=("fragmented", 0.3),
    old_topo=(2, 1), new_topo=(4, 1), role=(0, 0), seed=2,
    description="L40 H40 D128 bf16 bs16, 128 seqs lognormal(median 1500, cap 8192), 30% pre-occupied "
                "blocks, TP2/PP1 -> TP4/PP1",
)

GQA_70B = KVWorkload(
    name="gqa70b",
    num_layers=80, num_kv_heads=8, head_dim=128, elem_bytes=2, dtype="bf16",
    old_block_size=16, new_block_size=16,
    num_seqs=256, length_law=("lognormal", 2048, 0.5, 32768),
    pool_law=("slack", 1.1),
    old_topo=(8, 1), new_topo=(4, 2), role=(0, 0), seed=3,
    description="L80 H8 D128 bf16 bs16, 256 seqs lognormal(median 2048, cap 32768), TP8/PP1 -> TP4/PP2",
)

GQA_70B_LONG = KVWorkload(
    name="gqa70b_long",
    num_layers=80, num_kv_heads=8, head_dim=128, elem_bytes=2, dtype="bf16",
    old_block_size=16, new_block_size=32,
    num_seqs=8, length_law=("fixed", 131072),
    pool_law=("slack", 1.1),
    old_topo=(4, 2), new_topo=(8, 1), role=(0, 0), seed=4,
    description="L80 H8 D128 bf16, 8 x 131072 tokens, block size 16 -> 32, TP4/PP2 -> TP8/PP1",
)

QWEN3_30B = KVWorkload(
    name="qwen30b",
    num_layers=48, num_kv_heads=4, head_dim=128, elem_bytes=2, dtype="bf16",
    old_block_size=16, new_block_size=16,
    num_seqs=256, length_law=("lognormal", 2048, 0.5, 32768),
    pool_law=("slack", 1.1),
    old_topo=(8, 1), new_topo=(4, 2), role=(0, 0), seed=5,
    description="Qwen3-30B-A3B KV shape: L48 H4 D128 bf16 bs16, 256 seqs lognormal(median 2048, cap 32768), "
                "TP8/PP1 (each KV head on two ranks) -> TP4/PP2",
)

DS_32B = KVWorkload(
    name="ds32b",
    num_layers=64, num_kv_heads=8, head_dim=128, elem_bytes=2, dtype="bf16",
    old_block_size=16, new_block_size=16,
    num_seqs=256, length_law=("lognormal", 2048, 0.5, 32768),
    pool_law=("slack", 1.1),
    old_topo=(1, 8), new_topo=(4, 2), role=(0, 0), seed=6,
    description="DeepSeek-R1-Distill-Qwen-32B KV shape: L64 H8 D128 bf16 bs16, 256 seqs lognormal(median 2048, "
                "cap 32768), TP1/PP8 -> TP4/PP2",
)

WORKLOADS = {w.name: w for w in (TINY, MHA_7B, MHA_13B, GQA_70B, GQA_70B_LONG, QWEN3_30B, DS_32B)}


def reduced(w: KVWorkload, num_seqs: int = 5, max_len: int = 300, seed_offset: int = 100) -> KVWorkload:
    """Same shape, topology and pool law as `w`, with a small live population.

    Used by the many small parity cases (all ranks, edge cases, layouts, the
    CPU model of the kernels); the full-size populations are compared byte for
    byte in the full-size GPU tests.  The layer, head and block structure is
    unchanged, so a copy still spans many tiles and ends in partial blocks.
    """
    return w.replace(
        name=w.name + "_reduced",
        num_seqs=num_seqs,
        length_law=("uniform", 1, max_len),
        pool_law=w.pool_law if w.pool_law[0] != "fixed" else ("slack", 1.5),
        seed=w.seed + seed_offset,
    )
