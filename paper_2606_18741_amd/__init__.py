"""Two-dimensional KV-cache migration (ReMP, Section 3.4) and GPU shard rebuild
from a host weight store (Section 3.3) for MI355X / gfx950.

The work happens in libremp_kv.so (host planners + HIP kernels); this package is
its ctypes binding.  Importing it loads the library and fails loudly when the
library has not been built: there is no other execution path.
"""
from . import _lib
from ._lib import (EXPORTED, LAYOUT_HND, LAYOUT_NHD, LAYOUT_ROCM_SPLIT, REMP_KV_REUSE_DESCRIPTORS, REMP_KV_SKIP_LOCAL, STATUS, Buffer, DevTables, HostTables, Plan, PoolArg,
                   RempError, buffers, dev_tables, load, remp_kv_copy_local, remp_kv_pack, remp_kv_plan,
                   remp_kv_plan_destroy, remp_kv_plan_get_info, remp_kv_plan_get_pair, remp_kv_plan_query,
                   remp_kv_set_trace_events, remp_kv_unpack, remp_kv_unpack_noalloc, remp_kv_version, remp_kv_workspace_bytes,
                   remp_last_error, remp_status_string, REMP_W_COPY_ENGINE, REMP_W_FIRST_STAGE,
                   REMP_W_LAST_STAGE, REMP_W_REPLICATED, REMP_W_SPLIT_COLS, REMP_W_SPLIT_ROWS, WeightPlan,
                   WeightTensors, remp_w_load, remp_w_plan, remp_w_plan_destroy, remp_w_shard_bytes,
                   remp_w_shard_shape)

load()

__all__ = [
    "EXPORTED", "LAYOUT_HND", "LAYOUT_NHD", "LAYOUT_ROCM_SPLIT", "REMP_KV_REUSE_DESCRIPTORS", "REMP_KV_SKIP_LOCAL", "STATUS", "Buffer", "DevTables", "HostTables", "Plan", "PoolArg",
    "RempError", "buffers", "dev_tables", "load", "remp_kv_copy_local", "remp_kv_pack", "remp_kv_plan",
    "remp_kv_plan_destroy", "remp_kv_plan_get_info", "remp_kv_plan_get_pair", "remp_kv_plan_query",
    "remp_kv_set_trace_events", "remp_kv_unpack", "remp_kv_unpack_noalloc", "remp_kv_version", "remp_kv_workspace_bytes",
    "remp_last_error", "remp_status_string", "REMP_W_COPY_ENGINE", "REMP_W_FIRST_STAGE", "REMP_W_LAST_STAGE",
    "REMP_W_REPLICATED", "REMP_W_SPLIT_COLS", "REMP_W_SPLIT_ROWS", "WeightPlan", "WeightTensors", "remp_w_load",
    "remp_w_plan", "remp_w_plan_destroy", "remp_w_shard_bytes", "remp_w_shard_shape",
]
