"""Edge-case KV-migration configurations (inputs only), shared by the GPU parity tests and the CPU
model of the kernels."""
from __future__ import annotations

import numpy as np

import synthkv


def custom(**kw):
    base = dict(name="edge", num_layers=4, num_kv_heads=8, head_dim=64, elem_bytes=2, dtype="u16",
                old_block_size=16, new_block_size=16, num_seqs=6, length_law=("uniform", 0, 90),
                pool_law=("slack", 1.3), old_topo=(2, 1), new_topo=(1, 2), role="all", seed=21)
    base.update(kw)
    return synthkv.KVWorkload(**base)


EDGE = {
    "heads_not_nested_reblock": custom(num_layers=6, num_kv_heads=12, head_dim=32, old_topo=(3, 1),
                                        new_topo=(2, 3), old_block_size=8, new_block_size=16),
    "fp8_elements": custom(elem_bytes=1, old_topo=(4, 1), new_topo=(1, 4)),
    "fp32_elements": custom(elem_bytes=4, head_dim=16, old_topo=(1, 2), new_topo=(8, 1)),
    "odd_row_bytes": custom(num_kv_heads=4, head_dim=3, old_topo=(2, 1), new_topo=(4, 1)),
    "identity_2x2": custom(old_topo=(2, 2), new_topo=(2, 2)),
    "block_shrink_32_to_8": custom(old_block_size=32, new_block_size=8, old_topo=(1, 1), new_topo=(2, 2)),
    "non_power_of_two_block": custom(old_block_size=12, new_block_size=5, old_topo=(2, 2), new_topo=(4, 1)),
    "one_token": custom(num_seqs=1, length_law=("fixed", 1)),
    "long_single_sequence": custom(num_seqs=1, length_law=("fixed", 20011), num_layers=2, num_kv_heads=2,
                                   old_topo=(2, 1), new_topo=(1, 2), head_dim=128),
    "fragmented_pool": custom(pool_law=("fragmented", 0.5), num_seqs=12),
    "all_empty": custom(length_law=("fixed", 0)),
    "many_sequences": custom(num_seqs=1500, length_law=("uniform", 0, 9), num_layers=2),
    # GQA with more tensor ranks than KV heads (e.g. 4 KV heads at TP8): heads are replicated
    "replicated_tp8_to_tp2": custom(num_layers=8, num_kv_heads=4, head_dim=128, old_topo=(8, 1), new_topo=(2, 1)),
    "replicated_tp2pp2_to_tp8": custom(num_layers=8, num_kv_heads=4, head_dim=128, old_topo=(2, 2),
                                        new_topo=(8, 1)),
    "replicated_tp16_to_tp8pp2": custom(num_layers=8, num_kv_heads=4, head_dim=64, old_topo=(16, 1),
                                         new_topo=(8, 2), old_block_size=16, new_block_size=32),
    "replicated_keep_local": custom(num_layers=8, num_kv_heads=4, head_dim=128, old_topo=(8, 1), new_topo=(4, 2)),
    # several sources fill each new row with equal shares of >= 256 B: unpack writes whole rows (the fp8 case
    # below has four 512 B shares; heads_not_nested_reblock has unequal shares and takes per-slice copies)
    "merged_rows_mha": custom(num_layers=4, num_kv_heads=16, head_dim=128, old_topo=(4, 1), new_topo=(2, 2)),
    "merged_rows_reblock": custom(num_layers=4, num_kv_heads=32, head_dim=128, old_topo=(8, 1),
                                   new_topo=(2, 2), old_block_size=16, new_block_size=32),
    # several destinations split an old rank's rows into 256 B shares: pack reads whole rows
    "pack_rows_tp2_to_tp4": custom(num_layers=4, num_kv_heads=4, head_dim=128, old_topo=(2, 1), new_topo=(4, 1)),
    "pack_rows_4way_reblock": custom(num_layers=3, num_kv_heads=4, head_dim=128, old_topo=(1, 1),
                                      new_topo=(4, 1), old_block_size=16, new_block_size=32),
    "short_row_shares_fp8": custom(num_layers=4, num_kv_heads=32, head_dim=128, elem_bytes=1,
                                   old_topo=(8, 1), new_topo=(2, 2), old_block_size=16, new_block_size=32),
    # large blocks (128 -> 256 tokens: 128-512 KiB units, more than a workgroup's byte target)
    "large_blocks_reblock": custom(num_layers=2, num_kv_heads=8, head_dim=128, old_block_size=128,
                                   new_block_size=256, old_topo=(2, 1), new_topo=(1, 2),
                                   length_law=("uniform", 0, 2000)),
    # one KV head of 576 elements at every tensor rank (a compressed latent cache, replicated by
    # tensor parallelism): the extreme of replication, 1152-byte rows
    "replicated_single_latent_head": custom(num_layers=4, num_kv_heads=1, head_dim=576, old_topo=(4, 1),
                                           new_topo=(2, 2)),
    # explicit uneven pipeline partitions
    "uneven_pp": custom(num_layers=5, old_topo=(2, 2, (0, 3, 5)), new_topo=(1, 3, (0, 1, 2, 5))),
    "uneven_to_even": custom(num_layers=6, old_topo=(1, 4, (0, 1, 3, 4, 6)), new_topo=(2, 2),
                              new_block_size=32),
}


# The library's size limits: 2^31 - 2^20 live tokens (the plan takes at most 2^31 - 1) in 2048 sequences,
# re-blocked from 16 to 8 tokens per block, so the new tables hold 2^28 - 2^17 live blocks (the plan takes
# fewer than 2^28).  One 4-byte head row per token keeps each K or V pool at 8 GiB; one rank keeps everything.
LIMITS = custom(name="limits", num_layers=1, num_kv_heads=1, head_dim=4, elem_bytes=1, dtype="u8",
                old_block_size=16, new_block_size=8, num_seqs=2048, length_law=("fixed", (1 << 20) - (1 << 9)),
                pool_law=("slack", 1.001), old_topo=(1, 1), new_topo=(1, 1), role=(0, 0), seed=31)


# Pool layout pairs (old, new) and new block sizes of the shifted-lengths case: NHD, HND and ROCm tiles,
# same and mixed, with the old block size (16) kept or doubled.
SHIFTED_LAYOUTS = [(0, 0, 16), (1, 1, 16), (2, 2, 16), (0, 1, 16), (1, 1, 32), (2, 2, 32), (2, 0, 32)]


def shifted_old_lengths_case(new_block_size: int = 16):
    """Identity topology (every slice is local) and old device tables that disagree with the host ones:
    17 tokens move from sequence 1 to sequence 0 (same total, shifted starts), and sequence 1's first old
    block is physical block 0.  The local copies combine the new expansion's token offsets with the old
    one's, so the first 16 rows of sequence 1 get a negative token index.  Returns (workload, inputs,
    (device lengths, device row offsets, device block ids))."""
    w = custom(num_layers=2, num_kv_heads=8, head_dim=64, old_topo=(2, 1), new_topo=(2, 1), num_seqs=3,
               length_law=("fixed", 40), seed=5, new_block_size=new_block_size)
    inp = synthkv.make_inputs(w)
    t = inp.old_tables
    lens = t.seq_lens.copy()
    lens[0] += 17
    lens[1] -= 17
    ids = t.ids.copy()
    first1 = int(t.offsets[1])
    zero = np.nonzero(ids == 0)[0]
    if zero.size:
        ids[zero[0]], ids[first1] = ids[first1], 0
    else:
        ids[first1] = 0
    return w, inp, (lens, t.offsets.copy(), ids)
