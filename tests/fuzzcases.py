"""Seeded random KV-migration configurations for the GPU fuzz tests (inputs only)."""
from __future__ import annotations

import os

import numpy as np

import synthkv


def seed_range(default_stop: int):
    """Seeds of the random configurations: range(0, default_stop), or REMP_FUZZ_SEEDS="start:stop" to run
    another range of the same generator (longer runs outside the default suite)."""
    spec = os.environ.get("REMP_FUZZ_SEEDS")
    if spec:
        a, b = spec.split(":")
        return range(int(a), int(b))
    return range(default_stop)


def layout_count(default: int) -> int:
    """Number of layout cases: `default`, or REMP_FUZZ_LAYOUT_CASES."""
    return int(os.environ.get("REMP_FUZZ_LAYOUT_CASES", default))


def random_workload(seed: int) -> synthkv.KVWorkload:
    rng = np.random.default_rng(1000 + seed)
    L = int(rng.integers(1, 7))
    H = int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16]))
    e = int(rng.choice([1, 2, 4]))
    # head rows of any byte length that is a multiple of 4 (the generator fills 32-bit words)
    D = int(rng.choice({1: [4, 8, 12, 64, 128], 2: [2, 6, 8, 64, 128], 4: [1, 3, 16, 32]}[e]))

    def topo():
        tps = [t for t in range(1, 17) if H % t == 0 or t % H == 0]
        tp = int(rng.choice(tps))
        pp = int(rng.integers(1, min(L, max(1, 16 // tp), 4) + 1))
        if pp > 1 and (L % pp or rng.random() < 0.4):
            cuts = sorted(int(c) for c in rng.choice(np.arange(1, L), pp - 1, replace=False))
            return (tp, pp, tuple([0] + cuts + [L]))
        return (tp, pp)

    sizes = [1, 2, 3, 4, 8, 16, 32]
    if rng.random() < 0.5:
        pool = ("slack", float(rng.uniform(1.0, 2.0)))
    else:
        pool = ("fragmented", float(rng.uniform(0.1, 0.6)))
    return synthkv.KVWorkload(
        name=f"fuzz{seed}", num_layers=L, num_kv_heads=H, head_dim=D, elem_bytes=e, dtype="raw",
        old_block_size=int(rng.choice(sizes)), new_block_size=int(rng.choice(sizes)),
        num_seqs=int(rng.integers(0, 8)), length_law=("uniform", 0, int(rng.integers(1, 300))),
        pool_law=pool, old_topo=topo(), new_topo=topo(), role="all", seed=500 + seed)


def random_windows(seed: int, L: int):
    rng = np.random.default_rng(2000 + seed)
    k = int(rng.integers(0, min(L, 3)))
    cuts = sorted(int(c) for c in rng.choice(np.arange(1, L), k, replace=False)) if L > 1 and k else []
    b = [0] + cuts + [L]
    return list(zip(b[:-1], b[1:]))


LAYOUT_PAIRS = [(1, 1), (1, 2), (2, 1), (2, 2), (0, 1), (1, 0), (0, 2), (2, 0)]


def layout_cases(n: int, start: int = 40):
    """(seed, old layout, new layout) for the first n seeds from `start` whose shapes the head-tile
    layouts take (16-byte head rows; for the ROCm layout 16-byte block columns too); the layout pair of
    a seed is drawn from its own stream.  Layouts: 0 NHD, 1 HND, 2 ROCm."""
    out, seed = [], start
    while len(out) < n and seed < start + 20 * n:
        w = random_workload(seed)
        lo, ln = LAYOUT_PAIRS[np.random.default_rng(3000 + seed).integers(len(LAYOUT_PAIRS))]
        rocm_ok = all((bs * w.elem_bytes) % 16 == 0 for bs in (w.old_block_size, w.new_block_size))
        if (w.head_dim * w.elem_bytes) % 16 == 0 and (2 not in (lo, ln) or rocm_ok):
            out.append((seed, lo, ln))
        seed += 1
    return out
