"""ctypes binding of libremp_kv.so (include/remp_kv.h, include/remp_weights.h): argument marshalling only.

Every step of the migration runs in the library (host planner, HIP kernels);
this module converts Python values into the C structures and back.  Device
buffers are passed as integer addresses (e.g. torch.Tensor.data_ptr()) and
streams as raw HIP stream handles (torch.cuda.Stream.cuda_stream).
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, Structure, byref, c_char_p, c_int32, c_int64, c_void_p
from typing import Optional, Sequence, Tuple

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libremp_kv.so")

REMP_OK = 0
STATUS = {0: "REMP_OK", -1: "REMP_E_INVALID", -2: "REMP_E_UNSUPPORTED", -3: "REMP_E_RANGE",
          -4: "REMP_E_CAPACITY", -5: "REMP_E_ALIGN", -6: "REMP_E_SIZE", -7: "REMP_E_HIP"}

# every symbol include/remp_kv.h and include/remp_weights.h declare
EXPORTED = (
    "remp_kv_plan", "remp_kv_plan_destroy", "remp_kv_plan_get_info", "remp_kv_plan_get_pair",
    "remp_kv_plan_query", "remp_kv_workspace_bytes", "remp_kv_pack", "remp_kv_unpack", "remp_kv_unpack_noalloc",
    "remp_kv_copy_local",
    "remp_kv_set_trace_events", "remp_status_string", "remp_last_error", "remp_kv_version",
    "remp_w_plan", "remp_w_plan_destroy", "remp_w_shard_shape", "remp_w_shard_bytes", "remp_w_load",
)

REMP_KV_SKIP_LOCAL = 1
REMP_KV_REUSE_DESCRIPTORS = 2

# remp_weights.h
REMP_W_REPLICATED, REMP_W_SPLIT_ROWS, REMP_W_SPLIT_COLS = 0, 1, 2
REMP_W_FIRST_STAGE, REMP_W_LAST_STAGE = -1, -2
REMP_W_COPY_ENGINE = 1


class RempError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        self.status_name = STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.status_name}: {detail}")


class Topo(Structure):
    _fields_ = [("tp", c_int32), ("pp", c_int32), ("layer_starts", POINTER(c_int32))]


class Shape(Structure):
    _fields_ = [("num_layers", c_int32), ("num_kv_heads", c_int32), ("head_dim", c_int32),
                ("elem_bytes", c_int32), ("old_block_size", c_int32), ("new_block_size", c_int32)]


class BlockTables(Structure):
    _fields_ = [("num_seqs", c_int32), ("seq_lens", POINTER(c_int32)), ("row_offsets", POINTER(c_int32)),
                ("block_ids", POINTER(c_int32)), ("num_blocks", c_int64)]


class DevTables(Structure):
    _fields_ = [("seq_lens", c_void_p), ("row_offsets", c_void_p), ("block_ids", c_void_p)]


class Pool(Structure):
    _fields_ = [("num_layers", c_int32), ("layout", c_int32), ("k", POINTER(c_void_p)), ("v", POINTER(c_void_p)),
                ("num_blocks", c_int64)]


LAYOUT_NHD, LAYOUT_HND, LAYOUT_ROCM_SPLIT = 0, 1, 2


class Buffer(Structure):
    _fields_ = [("ptr", c_void_p), ("bytes", c_int64)]


class WPart(Structure):
    _fields_ = [("host", c_void_p), ("rows", c_int64), ("cols", c_int64), ("split", c_int32), ("units", c_int32)]


class WTensor(Structure):
    _fields_ = [("layer", c_int32), ("num_parts", c_int32), ("parts", POINTER(WPart))]


class PlanInfo(Structure):
    _fields_ = [("old_world", c_int32), ("new_world", c_int32), ("num_pairs", c_int32), ("num_items", c_int32),
                ("total_tokens", c_int64), ("old_live_blocks", c_int64), ("new_live_blocks", c_int64)]


class PairInfo(Structure):
    _fields_ = [("src", c_int32), ("dst", c_int32), ("layer_begin", c_int32), ("layer_end", c_int32),
                ("head_begin", c_int32), ("head_count", c_int32), ("slice_bytes", c_int64),
                ("staging_bytes", c_int64)]


_lib = None


def load(path: str = _LIB_PATH) -> ctypes.CDLL:
    """Load the library (once).  Raises ImportError if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python paper_2606_18741_amd/build.py` "
                          "(the migration has no fallback path)")
    # torch carries its own HIP runtime.  Loading torch first lets the library's
    # libamdhip64.so.7 dependency resolve to that same runtime, so device
    # pointers, streams and events are shared by one runtime in the process.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    runtimes = _mapped_hip_runtimes()
    if len(runtimes) > 1:
        raise ImportError("more than one HIP runtime is loaded in this process "
                          f"({', '.join(runtimes)}); import torch before anything else that loads HIP")
    st = c_int32
    lib.remp_kv_plan.argtypes = [POINTER(Topo), POINTER(Topo), POINTER(Shape), POINTER(BlockTables),
                                 POINTER(c_void_p)]
    lib.remp_kv_plan.restype = st
    lib.remp_kv_plan_destroy.argtypes = [c_void_p]
    lib.remp_kv_plan_destroy.restype = None
    lib.remp_kv_plan_get_info.argtypes = [c_void_p, POINTER(PlanInfo)]
    lib.remp_kv_plan_get_info.restype = st
    lib.remp_kv_plan_get_pair.argtypes = [c_void_p, c_int32, POINTER(PairInfo)]
    lib.remp_kv_plan_get_pair.restype = st
    lib.remp_kv_plan_query.argtypes = [c_void_p, c_int32, c_int32, POINTER(c_int64), POINTER(c_int64)]
    lib.remp_kv_plan_query.restype = st
    lib.remp_kv_workspace_bytes.argtypes = [c_void_p, POINTER(c_int64)]
    lib.remp_kv_workspace_bytes.restype = st
    lib.remp_kv_pack.argtypes = [c_void_p, c_int32, c_int32, c_int32, POINTER(Pool), POINTER(DevTables),
                                 POINTER(Buffer), c_void_p, c_int64, ctypes.c_uint32, c_void_p]
    lib.remp_kv_pack.restype = st
    lib.remp_kv_unpack.argtypes = [c_void_p, c_int32, c_int32, c_int32, POINTER(Buffer), POINTER(Pool),
                                   POINTER(BlockTables), POINTER(DevTables), c_void_p, c_int64, ctypes.c_uint32,
                                   c_void_p]
    lib.remp_kv_unpack.restype = st
    lib.remp_kv_unpack_noalloc.argtypes = [c_void_p, c_int32, c_int32, c_int32, POINTER(Buffer), POINTER(Pool),
                                           POINTER(BlockTables), POINTER(DevTables), c_void_p, ctypes.c_uint32,
                                           c_void_p]
    lib.remp_kv_unpack_noalloc.restype = st
    lib.remp_kv_copy_local.argtypes = [c_void_p, c_int32, c_int32, c_int32, POINTER(Pool), POINTER(DevTables),
                                       POINTER(Pool), POINTER(BlockTables), POINTER(DevTables), c_void_p, c_int64,
                                       ctypes.c_uint32, c_void_p]
    lib.remp_kv_copy_local.restype = st
    lib.remp_kv_set_trace_events.argtypes = [c_void_p, c_void_p]
    lib.remp_kv_set_trace_events.restype = None
    lib.remp_w_plan.argtypes = [POINTER(Topo), c_int32, c_int32, POINTER(WTensor), c_int32, POINTER(c_void_p)]
    lib.remp_w_plan.restype = st
    lib.remp_w_plan_destroy.argtypes = [c_void_p]
    lib.remp_w_plan_destroy.restype = None
    lib.remp_w_shard_shape.argtypes = [c_void_p, c_int32, c_int32, POINTER(c_int64), POINTER(c_int64)]
    lib.remp_w_shard_shape.restype = st
    lib.remp_w_shard_bytes.argtypes = [c_void_p, c_int32, c_int32, c_int32, POINTER(c_int64)]
    lib.remp_w_shard_bytes.restype = st
    lib.remp_w_load.argtypes = [c_void_p, c_int32, c_int32, c_int32, POINTER(c_void_p), ctypes.c_uint32, c_int32,
                                c_void_p]
    lib.remp_w_load.restype = st
    lib.remp_status_string.argtypes = [c_int32]
    lib.remp_status_string.restype = c_char_p
    lib.remp_last_error.argtypes = []
    lib.remp_last_error.restype = c_char_p
    lib.remp_kv_version.argtypes = []
    lib.remp_kv_version.restype = c_char_p
    _lib = lib
    return lib


def _mapped_hip_runtimes():
    """Distinct libamdhip64 files mapped into this process (Linux)."""
    try:
        with open("/proc/self/maps") as f:
            return sorted({os.path.realpath(ln.split()[-1]) for ln in f if "libamdhip64" in ln})
    except OSError:
        return []


def _check(status: int, where: str) -> None:
    if status != REMP_OK:
        raise RempError(status, where, load().remp_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(x) -> Optional[int]:
    """Device address of an int, None or object with data_ptr()."""
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    return int(x)


def _ref(x):
    """byref of a wrapper's C struct (or of a ctypes struct); None stays NULL."""
    if x is None:
        return None
    return byref(x.c) if hasattr(x, "c") else byref(x)


class HostTables:
    """Host block tables kept alive for the duration of C calls."""

    def __init__(self, seq_lens, row_offsets, block_ids, num_blocks: int):
        self.seq_lens = _i32(seq_lens)
        self.row_offsets = _i32(row_offsets)
        self.block_ids = _i32(block_ids) if len(block_ids) else np.zeros(1, dtype=np.int32)
        self.num_blocks = int(num_blocks)
        self.c = BlockTables(
            int(self.seq_lens.shape[0]),
            self.seq_lens.ctypes.data_as(POINTER(c_int32)),
            self.row_offsets.ctypes.data_as(POINTER(c_int32)),
            self.block_ids.ctypes.data_as(POINTER(c_int32)),
            self.num_blocks)

    @classmethod
    def of(cls, t) -> "HostTables":
        """From any object with seq_lens, offsets, ids, num_blocks (e.g. synthkv.BlockTables)."""
        return cls(t.seq_lens, t.offsets, t.ids, t.num_blocks)


def dev_tables(seq_lens, row_offsets, block_ids) -> DevTables:
    return DevTables(_ptr(seq_lens), _ptr(row_offsets), _ptr(block_ids))


class PoolArg:
    """A rank's paged storage: K and V device addresses per local layer (None allowed)."""

    def __init__(self, k: Sequence, v: Sequence, num_blocks: int, layout: int = LAYOUT_NHD):
        assert len(k) == len(v)
        n = len(k)
        self._k = (c_void_p * max(n, 1))(*[_ptr(x) for x in k])
        self._v = (c_void_p * max(n, 1))(*[_ptr(x) for x in v])
        self.c = Pool(n, int(layout), ctypes.cast(self._k, POINTER(c_void_p)),
                      ctypes.cast(self._v, POINTER(c_void_p)), int(num_blocks))


def buffers(entries: Sequence[Optional[Tuple[object, int]]]):
    """Array of remp_buffer from [(address_or_tensor, bytes) | None, ...]."""
    arr = (Buffer * max(len(entries), 1))()
    for i, e in enumerate(entries):
        if e is None:
            arr[i] = Buffer(None, 0)
        else:
            arr[i] = Buffer(_ptr(e[0]), int(e[1]))
    return arr


# ---------------------------------------------------------------------------
# the C entry points under their own names
# ---------------------------------------------------------------------------

def _topo(t):
    """(tp, pp) or (tp, pp, layer_starts) -> (Topo, keep-alive array)."""
    starts = None
    if len(t) > 2 and t[2] is not None:
        starts = _i32(t[2])
        return Topo(int(t[0]), int(t[1]), starts.ctypes.data_as(POINTER(c_int32))), starts
    return Topo(int(t[0]), int(t[1]), None), starts


def remp_kv_plan(old_topo, new_topo, shape: Tuple[int, ...], old_tables: HostTables) -> c_void_p:
    """Topologies are (tp, pp) or (tp, pp, layer_starts[pp + 1]);
    shape = (num_layers, num_kv_heads, head_dim, elem_bytes, old_block_size, new_block_size)."""
    lib = load()
    out = c_void_p()
    ot, keep_o = _topo(old_topo)
    nt, keep_n = _topo(new_topo)
    _check(lib.remp_kv_plan(byref(ot), byref(nt), byref(Shape(*shape)), byref(old_tables.c), byref(out)),
           "remp_kv_plan")
    return out


def remp_kv_plan_destroy(plan) -> None:
    load().remp_kv_plan_destroy(plan)


def remp_kv_plan_get_info(plan) -> PlanInfo:
    info = PlanInfo()
    _check(load().remp_kv_plan_get_info(plan, byref(info)), "remp_kv_plan_get_info")
    return info


def remp_kv_plan_get_pair(plan, index: int) -> PairInfo:
    p = PairInfo()
    _check(load().remp_kv_plan_get_pair(plan, index, byref(p)), "remp_kv_plan_get_pair")
    return p


def remp_kv_plan_query(plan, src: int, dst: int, num_layers: int) -> Tuple[int, np.ndarray]:
    nbytes = c_int64()
    offs = np.zeros(num_layers + 1, dtype=np.int64)
    _check(load().remp_kv_plan_query(plan, src, dst, byref(nbytes), offs.ctypes.data_as(POINTER(c_int64))),
           "remp_kv_plan_query")
    return int(nbytes.value), offs


def remp_kv_workspace_bytes(plan) -> int:
    n = c_int64()
    _check(load().remp_kv_workspace_bytes(plan, byref(n)), "remp_kv_workspace_bytes")
    return int(n.value)


def remp_kv_pack(plan, old_rank: int, layer_begin: int, layer_end: int, src: PoolArg, old_dev_tables: DevTables,
                 staging, workspace, workspace_bytes: int, flags: int, stream: int) -> None:
    _check(load().remp_kv_pack(plan, old_rank, layer_begin, layer_end, _ref(src), _ref(old_dev_tables),
                               staging, _ptr(workspace), int(workspace_bytes), int(flags), c_void_p(stream)),
           "remp_kv_pack")


def remp_kv_unpack(plan, new_rank: int, layer_begin: int, layer_end: int, staging, dst: PoolArg,
                   new_tables: HostTables, new_dev_tables: DevTables, workspace, workspace_bytes: int,
                   flags: int, stream: int) -> None:
    _check(load().remp_kv_unpack(plan, new_rank, layer_begin, layer_end, staging, _ref(dst),
                                 _ref(new_tables), _ref(new_dev_tables), _ptr(workspace),
                                 int(workspace_bytes), int(flags), c_void_p(stream)), "remp_kv_unpack")


def remp_kv_unpack_noalloc(plan, new_rank: int, layer_begin: int, layer_end: int, staging, dst: PoolArg,
                           new_tables: HostTables, new_dev_tables: DevTables, status, flags: int,
                           stream: int) -> None:
    _check(load().remp_kv_unpack_noalloc(plan, new_rank, layer_begin, layer_end, staging, _ref(dst),
                                         _ref(new_tables), _ref(new_dev_tables), _ptr(status), int(flags),
                                         c_void_p(stream)), "remp_kv_unpack_noalloc")


def remp_kv_copy_local(plan, rank: int, layer_begin: int, layer_end: int, src: PoolArg, old_dev_tables: DevTables,
                       dst: PoolArg, new_tables: HostTables, new_dev_tables: DevTables, workspace,
                       workspace_bytes: int, flags: int, stream: int) -> None:
    _check(load().remp_kv_copy_local(plan, rank, layer_begin, layer_end, _ref(src), _ref(old_dev_tables),
                                     _ref(dst), _ref(new_tables), _ref(new_dev_tables), _ptr(workspace),
                                     int(workspace_bytes), int(flags), c_void_p(stream)), "remp_kv_copy_local")


def remp_kv_set_trace_events(start: Optional[int], stop: Optional[int]) -> None:
    load().remp_kv_set_trace_events(start, stop)


def remp_status_string(status: int) -> str:
    return load().remp_status_string(status).decode()


def remp_last_error() -> str:
    return load().remp_last_error().decode()


def remp_kv_version() -> str:
    return load().remp_kv_version().decode()


# --- weight shards (remp_weights.h) ---------------------------------------

class WeightTensors:
    """C arrays of remp_w_tensor / remp_w_part for a list of tensors.

    tensors: sequence of (layer, parts); parts: sequence of
    (host_address, rows, cols, split, units).  Keeps the arrays alive.
    """

    def __init__(self, tensors):
        self.part_arrays = []
        arr = (WTensor * max(1, len(tensors)))()
        for i, (layer, parts) in enumerate(tensors):
            pa = (WPart * len(parts))(*[WPart(int(h) if h else None, int(r), int(c), int(sp), int(u))
                                        for (h, r, c, sp, u) in parts])
            self.part_arrays.append(pa)
            arr[i] = WTensor(int(layer), len(parts), ctypes.cast(pa, POINTER(WPart)))
        self.array = arr
        self.count = len(tensors)


def remp_w_plan(topo, num_layers: int, elem_bytes: int, tensors: WeightTensors) -> c_void_p:
    """topo = (tp, pp) or (tp, pp, layer_starts)."""
    lib = load()
    out = c_void_p()
    t, keep = _topo(topo)
    _check(lib.remp_w_plan(byref(t), int(num_layers), int(elem_bytes), tensors.array, tensors.count, byref(out)),
           "remp_w_plan")
    return out


def remp_w_plan_destroy(plan) -> None:
    load().remp_w_plan_destroy(plan)


def remp_w_shard_shape(plan, rank: int, tensor: int) -> Tuple[int, int]:
    r, c = c_int64(), c_int64()
    _check(load().remp_w_shard_shape(plan, int(rank), int(tensor), byref(r), byref(c)), "remp_w_shard_shape")
    return int(r.value), int(c.value)


def remp_w_shard_bytes(plan, rank: int, tensor_begin: int, tensor_end: int) -> int:
    b = c_int64()
    _check(load().remp_w_shard_bytes(plan, int(rank), int(tensor_begin), int(tensor_end), byref(b)),
           "remp_w_shard_bytes")
    return int(b.value)


def remp_w_load(plan, rank: int, tensor_begin: int, tensor_end: int, dst: Sequence, flags: int,
                max_workgroups: int, stream) -> None:
    """dst: one device address (int, tensor or None) per tensor index."""
    arr = (c_void_p * max(1, len(dst)))(*[_ptr(d) for d in dst])
    _check(load().remp_w_load(plan, int(rank), int(tensor_begin), int(tensor_end), arr, int(flags),
                              int(max_workgroups), c_void_p(stream)), "remp_w_load")


class WeightPlan:
    """Owns a remp_w_plan_t; the same calls with the plan bound."""

    def __init__(self, topo, num_layers: int, elem_bytes: int, tensors):
        self.tensors = tensors if isinstance(tensors, WeightTensors) else WeightTensors(tensors)
        self.num_tensors = self.tensors.count
        self.elem_bytes = int(elem_bytes)
        self.world = int(topo[0]) * int(topo[1])
        self.handle = remp_w_plan(topo, num_layers, elem_bytes, self.tensors)

    def close(self) -> None:
        if self.handle:
            remp_w_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def shard_shape(self, rank: int, tensor: int) -> Tuple[int, int]:
        return remp_w_shard_shape(self.handle, rank, tensor)

    def shard_bytes(self, rank: int, tensor_begin: int = 0, tensor_end: Optional[int] = None) -> int:
        return remp_w_shard_bytes(self.handle, rank, tensor_begin, self.num_tensors if tensor_end is None else tensor_end)

    def load(self, rank: int, dst: Sequence, stream, tensor_begin: int = 0, tensor_end: Optional[int] = None,
             flags: int = 0, max_workgroups: int = 0) -> None:
        remp_w_load(self.handle, rank, tensor_begin, self.num_tensors if tensor_end is None else tensor_end, dst,
                    flags, max_workgroups, stream)


# ---------------------------------------------------------------------------
# convenience owner of a plan handle
# ---------------------------------------------------------------------------

class Plan:
    """Owns a remp_kv_plan_t; the same calls with the plan bound."""

    def __init__(self, old_topo, new_topo, shape, old_tables: HostTables):
        self.shape = tuple(int(x) for x in shape)
        self.num_layers = self.shape[0]
        self.handle = remp_kv_plan(old_topo, new_topo, self.shape, old_tables)
        self.info = remp_kv_plan_get_info(self.handle)
        self.pairs = [remp_kv_plan_get_pair(self.handle, i) for i in range(self.info.num_pairs)]

    def close(self) -> None:
        if self.handle:
            remp_kv_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def query(self, src: int, dst: int) -> Tuple[int, np.ndarray]:
        return remp_kv_plan_query(self.handle, src, dst, self.num_layers)

    @property
    def workspace_bytes(self) -> int:
        return remp_kv_workspace_bytes(self.handle)

    def pack(self, old_rank, src: PoolArg, old_dev_tables: DevTables, staging, workspace, workspace_bytes,
             stream, layer_begin: int = 0, layer_end: Optional[int] = None, flags: int = 0) -> None:
        remp_kv_pack(self.handle, old_rank, layer_begin, self.num_layers if layer_end is None else layer_end,
                     src, old_dev_tables, staging, workspace, workspace_bytes, flags, stream)

    def unpack(self, new_rank, staging, dst: PoolArg, new_tables: HostTables, new_dev_tables: DevTables,
               workspace, workspace_bytes, stream, layer_begin: int = 0, layer_end: Optional[int] = None,
               flags: int = 0) -> None:
        remp_kv_unpack(self.handle, new_rank, layer_begin, self.num_layers if layer_end is None else layer_end,
                       staging, dst, new_tables, new_dev_tables, workspace, workspace_bytes, flags, stream)

    def unpack_noalloc(self, new_rank, staging, dst: PoolArg, new_tables: HostTables, new_dev_tables: DevTables,
                       status, stream, layer_begin: int = 0, layer_end: Optional[int] = None,
                       flags: int = 0) -> None:
        remp_kv_unpack_noalloc(self.handle, new_rank, layer_begin, self.num_layers if layer_end is None else layer_end,
                               staging, dst, new_tables, new_dev_tables, status, flags, stream)

    def copy_local(self, rank, src: PoolArg, old_dev_tables: DevTables, dst: PoolArg, new_tables: HostTables,
                   new_dev_tables: DevTables, workspace, workspace_bytes, stream, layer_begin: int = 0,
                   layer_end: Optional[int] = None, flags: int = 0) -> None:
        remp_kv_copy_local(self.handle, rank, layer_begin, self.num_layers if layer_end is None else layer_end,
                           src, old_dev_tables, dst, new_tables, new_dev_tables, workspace, workspace_bytes, flags,
                           stream)
