"""Two-dimensional KV-cache migration (ReMP, Section 3.4) for MI355X / gfx950.

The work happens in libremp_kv.so (host planner + HIP kernels); this package is
its ctypes binding.  Importing it loads the library and fails loudly when the
library has not been built: there is no other execution path.
"""
from . import _lib
from ._lib import (EXPORTED, LAYOUT_HND, LAYOUT_NHD, LAYOUT_ROCM_SPLIT, REMP_KV_SKIP_LOCAL, STATUS, Buffer, DevTables, HostTables, Plan, PoolArg,
                   RempError, buffers, dev_tables, load, remp_kv_copy_local, remp_kv_pack, remp_kv_plan,
                   remp_kv_plan_destroy, remp_kv_plan_get_info, remp_kv_plan_get_pair, remp_kv_plan_query,
                   remp_kv_set_trace_events, remp_kv_unpack, remp_kv_version, remp_kv_workspace_bytes,
                   remp_last_error, remp_status_string)

load()

__all__ = [
    "EXPORTED", "LAYOUT_HND", "LAYOUT_NHD", "LAYOUT_ROCM_SPLIT", "REMP_KV_SKIP_LOCAL", "STATUS", "Buffer", "DevTables", "HostTables", "Plan", "PoolArg",
    "RempError", "buffers", "dev_tables", "load", "remp_kv_copy_local", "remp_kv_pack", "remp_kv_plan",
    "remp_kv_plan_destroy", "remp_kv_plan_get_info", "remp_kv_plan_get_pair", "remp_kv_plan_query",
    "remp_kv_set_trace_events", "remp_kv_unpack", "remp_kv_version", "remp_kv_workspace_bytes",
    "remp_last_error", "remp_status_string",
]
