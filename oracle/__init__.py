"""CPU oracle for the KV-cache migration and the weight-shard rebuild.  TEST
INFRASTRUCTURE: only the tests, the smoke check and the benchmark's
CPU-baseline leg may use it."""
from .migration import (Topology, check_divisible, pp_owner, rank_of, layers_of,
                      heads_of, pair_slices, staging_bytes, token_slots, token_offsets, gather_rows,
                      holders, source_of, tp_owners,
                      reshard, staging_buffer, old_location, new_location, staging_location,
                      NHD, HND, ROCM_SPLIT, encode_pool, decode_pool)
from . import weights
