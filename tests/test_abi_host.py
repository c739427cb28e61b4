"""Host-side tests of libremp_kv.so through its C ABI (no GPU needed).

* the library loads and exports every function include/*.h declares;
* the planner's pairs, item counts, staging sizes and layer offsets equal the
  oracle's definition-based grouping and closed forms, over many topologies;
* every validation error is reported with its status before anything is
  enqueued.  Calls that must fail validation use stand-in addresses; they are
  skipped when a GPU is visible, so a validation bug could never launch a
  kernel on stand-in addresses.
"""
from __future__ import annotations

import ctypes
import itertools
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import paper_2606_18741_amd as rk
import synthkv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
T = oracle.Topology


def _divisors(n):
    return [d for d in range(1, n + 1) if n % d == 0]


def _has_gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


cpu_only = pytest.mark.skipif(_has_gpu(), reason="stand-in device addresses are only used without a GPU")


# ---------------------------------------------------------------------------
# exports
# ---------------------------------------------------------------------------

def test_exports_every_declared_symbol():
    import glob
    declared = []
    for path in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        with open(path) as f:
            declared += re.findall(r"REMP_API\s+[\w\s\*]+?\b(remp_\w+)\s*\(", f.read())
    assert len(declared) == len(set(declared)) >= 18
    lib = rk.load()
    for name in declared:
        assert hasattr(lib, name), f"{name} declared but not exported"
    assert set(declared) == set(rk.EXPORTED)
    assert rk.remp_kv_version().count(".") == 2
    for code, name in rk.STATUS.items():
        assert rk.remp_status_string(code) == name


def test_probe_library_exports_and_refuses_bad_arguments():
    """libremp_probe.so (HBM access-pattern probes, measurement only) exports its two entry points and refuses
    invalid arguments before touching the GPU."""
    import ctypes
    import subprocess
    path = os.path.join(os.path.dirname(rk._lib._LIB_PATH), "libremp_probe.so")
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True).stdout
    assert {ln.split()[-1] for ln in out.splitlines() if "remp_" in ln} == {"remp_probe_chunks", "remp_probe_phased"}
    fn = ctypes.CDLL(path).remp_probe_chunks
    fn.restype = ctypes.c_int32
    fn.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_void_p]
    ok = (0, 1 << 40, 1 << 41, None, 0, 16, 4096, None, None, 256, 2, 1, None)
    for i, bad in ((0, 4), (0, -1), (6, 4000), (9, 128), (10, 3), (11, 0), (5, 0)):
        a = list(ok)
        a[i] = bad
        assert fn(*a) == -1, (i, bad)
    ph = ctypes.CDLL(path).remp_probe_phased
    ph.restype = ctypes.c_int32
    ph.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_int32, ctypes.c_int32, ctypes.c_double, ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p]
    resident = ctypes.c_int32(-1)
    ok = [1 << 40, 1 << 41, 1 << 42, 1 << 30, 256, 8, 1, 256, 200.0, ctypes.byref(resident), None]
    for i, bad in ((4, 128), (5, 3), (6, 3), (6, -1)):   # refused before any HIP call
        a = list(ok)
        a[i] = bad
        assert ph(*a) == -1, (i, bad)
        assert resident.value == 0


def test_noalloc_refusals_before_any_device_call():
    """remp_kv_unpack_noalloc validates before it touches a device: a plan whose workspace exceeds the static
    scratch (REMP_E_SIZE), a misaligned status word (REMP_E_ALIGN) and a rank outside the new topology
    (REMP_E_RANGE) are refused on a machine without a GPU."""
    n = 1 << 22                                     # one sequence, 262144 blocks of 16 tokens
    big = rk.HostTables(np.array([n], np.int32), np.array([0, n // 16], np.int32),
                        np.arange(n // 16, dtype=np.int32), n // 16)
    plan = rk.Plan((1, 1), (1, 1), (1, 1, 8, 2, 16, 16), big)
    assert plan.workspace_bytes > 8 << 20           # REMP_KV_NOALLOC_SCRATCH_BYTES
    none_pool = lambda nb: rk.PoolArg([None], [None], nb)
    with pytest.raises(rk.RempError) as e:
        plan.unpack_noalloc(0, rk.buffers([None]), none_pool(n // 16), big, rk.dev_tables(None, None, None), None, 0)
    assert e.value.status_name == "REMP_E_SIZE"
    small = rk.HostTables(np.array([37], np.int32), np.array([0, 3], np.int32), np.array([5, 0, 2], np.int32), 8)
    plan = rk.Plan((1, 1), (1, 1), (1, 1, 8, 2, 16, 16), small)
    with pytest.raises(rk.RempError) as e:
        plan.unpack_noalloc(0, rk.buffers([None]), none_pool(8), small, rk.dev_tables(None, None, None), 0x1002, 0)
    assert e.value.status_name == "REMP_E_ALIGN"
    with pytest.raises(rk.RempError) as e:
        plan.unpack_noalloc(1, rk.buffers([None]), none_pool(8), small, rk.dev_tables(None, None, None), None, 0)
    assert e.value.status_name == "REMP_E_RANGE"


def test_tile_shape_refusals_before_any_device_call():
    """A (block, head) tile that does not fit the head-tile kernels' LDS budget (128 rows of 256 bytes, 34816
    bytes with the row padding) is refused by pack (ROCm pool), unpack and the local copy (HND pools) with
    REMP_E_UNSUPPORTED before anything is enqueued: no device is touched on a machine without a GPU.  (An
    HND pack whose slices carry one head each copies rows, not tiles, hence the ROCm pool for the pack.)"""
    tables = synthkv.tables_from_rows(np.array([300, 129], np.int32), [[3, 0, 5], [1, 6]], 8, 128)
    ht = rk.HostTables.of(tables)
    plan = rk.Plan((1, 1), (1, 1), (1, 1, 128, 2, 128, 128), ht)
    (pair,) = plan.pairs
    dev = rk.dev_tables(0x70000000, 0x70001000, 0x70002000)
    stage = rk.buffers([(0x50000000, pair.staging_bytes)])
    ws, ws_bytes = 0x60000000, plan.workspace_bytes
    src = lambda layout: rk.PoolArg([0x10000000], [0x20000000], 8, layout=layout)
    dst = lambda layout: rk.PoolArg([0x30000000], [0x40000000], 8, layout=layout)
    calls = {"pack": lambda: plan.pack(0, src(rk.LAYOUT_ROCM_SPLIT), dev, stage, ws, ws_bytes, None),
             "unpack": lambda: plan.unpack(0, stage, dst(rk.LAYOUT_HND), ht, dev, ws, ws_bytes, None),
             "local": lambda: plan.copy_local(0, src(rk.LAYOUT_HND), dev, dst(rk.LAYOUT_HND), ht, dev, ws, ws_bytes,
                                              None)}
    for name, call in calls.items():
        with pytest.raises(rk.RempError) as e:
            call()
        assert e.value.status_name == "REMP_E_UNSUPPORTED", name
        assert "LDS" in str(e.value), name


def test_only_the_abi_is_exported_from_host_code():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", rk._lib._LIB_PATH], capture_output=True, text=True).stdout
    names = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    abi = {n for n in names if n.startswith("remp_")}
    assert abi == set(rk.EXPORTED)


# ---------------------------------------------------------------------------
# the plan against the definition
# ---------------------------------------------------------------------------

def _tables(S=3, n=37, bs=16, N=64, seed=0):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, n, size=S).astype(np.int32)
    rows = []
    free = list(rng.permutation(N))
    for L_ in lens:
        k = (int(L_) + bs - 1) // bs
        rows.append(free[:k])
        free = free[k:]
    return synthkv.tables_from_rows(lens, rows, N, bs)


def _plan(old, new, L, H, D=8, e=2, bs_o=16, bs_n=16, tables=None):
    tables = tables if tables is not None else _tables(bs=bs_o)
    return rk.Plan(old, new, (L, H, D, e, bs_o, bs_n), rk.HostTables.of(tables)), tables


def _check_plan(old, new, L, H, D=8, e=2):
    p, tables = _plan(old, new, L, H, D, e)
    Tk = int(tables.seq_lens.sum())
    want = oracle.pair_slices(T(*old), T(*new), L, H)
    got = {(q.src, q.dst): (list(range(q.layer_begin, q.layer_end)),
                            list(range(q.head_begin, q.head_begin + q.head_count))) for q in p.pairs}
    assert got == want
    sizes = oracle.staging_bytes(T(*old), T(*new), L, H, D, e, Tk)
    for q in p.pairs:
        assert q.staging_bytes == sizes[(q.src, q.dst)]
        nbytes, offs = p.query(q.src, q.dst)
        assert nbytes == q.staging_bytes
        ls = want[(q.src, q.dst)][0]
        for l in range(L + 1):
            assert offs[l] == sum(1 for x in ls if x < l) * q.slice_bytes
    # pairs that exchange nothing report zero bytes
    for r in range(T(*old).world):
        for q in range(T(*new).world):
            if (r, q) not in want:
                assert p.query(r, q)[0] == 0
    # Algorithm 1 emits one item per (layer, new tensor rank, old tensor rank) with overlapping heads;
    # with replicated old heads, one per (layer, new tensor rank, target head) from the chosen replica
    def head_range(t, tp):
        return (t * H // tp, t * H // tp + 1) if tp > H else (t * H // tp, (t + 1) * H // tp)
    items = 0
    for l in range(L):
        for ntp in range(new[0]):
            a0, a1 = head_range(ntp, new[0])
            if old[0] > H:
                items += a1 - a0
                continue
            for otp in range(old[0]):
                b0, b1 = head_range(otp, old[0])
                items += max(a0, b0) < min(a1, b1)
    assert p.info.num_items == items == sum(q.layer_end - q.layer_begin for q in p.pairs)
    assert p.info.old_world == old[0] * old[1] and p.info.new_world == new[0] * new[1]
    assert p.info.total_tokens == Tk


def _tps(H, k=5):
    return _divisors(H)[:k] + [2 * H, 4 * H]


@pytest.mark.parametrize("L,H,tps", [(4, 8, None), (6, 12, None), (8, 8, None), (80, 8, None), (48, 4, None),
                                     (4, 1, None), (32, 32, [1, 2, 4, 8, 64]), (40, 40, [1, 2, 4, 8, 80])])
def test_plan_matches_definition(L, H, tps):
    tps = tps or _tps(H)
    for tp_o, pp_o, tp_n, pp_n in itertools.product(tps, _divisors(L)[:3], tps, _divisors(L)[:3]):
        _check_plan((tp_o, pp_o), (tp_n, pp_n), L, H)


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 12), st.integers(1, 12), st.data())
def test_plan_matches_definition_random(L, H, data):
    old = (data.draw(st.sampled_from(_tps(H, 99))), data.draw(st.sampled_from(_divisors(L))))
    new = (data.draw(st.sampled_from(_tps(H, 99))), data.draw(st.sampled_from(_divisors(L))))
    _check_plan(old, new, L, H, D=data.draw(st.integers(1, 9)), e=data.draw(st.sampled_from([1, 2, 4])))


@pytest.mark.parametrize("name", list(synthkv.WORKLOADS))
def test_workload_plans(name):
    w = synthkv.WORKLOADS[name]
    inp = synthkv.make_inputs(w)
    p = rk.Plan(w.old_topo, w.new_topo, (w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes,
                                         w.old_block_size, w.new_block_size), rk.HostTables.of(inp.old_tables))
    assert p.info.total_tokens == int(inp.lens.sum())
    nb = lambda bs: int(((inp.lens.astype(np.int64) + bs - 1) // bs).sum())
    assert p.info.old_live_blocks == nb(w.old_block_size)
    assert p.info.new_live_blocks == nb(w.new_block_size)
    sizes = oracle.staging_bytes(T(*w.old_topo), T(*w.new_topo), w.num_layers, w.num_kv_heads, w.head_dim,
                                 w.elem_bytes, int(inp.lens.sum()))
    assert {(q.src, q.dst): q.staging_bytes for q in p.pairs} == sizes
    assert p.workspace_bytes >= 16 * max(p.info.old_live_blocks, p.info.new_live_blocks)


# ---------------------------------------------------------------------------
# plan validation
# ---------------------------------------------------------------------------

def _expect(status, fn, *a, **k):
    with pytest.raises(rk.RempError) as ei:
        fn(*a, **k)
    assert ei.value.status_name == status, str(ei.value)
    assert rk.remp_last_error()
    return ei.value


def test_plan_errors():
    t = _tables()
    ht = rk.HostTables.of(t)
    shape = (4, 8, 8, 2, 16, 16)
    _expect("REMP_E_UNSUPPORTED", rk.Plan, (3, 1), (1, 1), shape, ht)        # H % TP and TP % H
    _expect("REMP_E_UNSUPPORTED", rk.Plan, (12, 1), (1, 1), shape, ht)
    _expect("REMP_E_UNSUPPORTED", rk.Plan, (1, 1), (1, 3), shape, ht)        # L % PP
    _expect("REMP_E_INVALID", rk.Plan, (0, 1), (1, 1), shape, ht)
    _expect("REMP_E_INVALID", rk.Plan, (1, 1), (1, 1), (4, 8, 8, 3, 16, 16), ht)   # elem bytes
    _expect("REMP_E_INVALID", rk.Plan, (1, 1), (1, 1), (4, 8, 0, 2, 16, 16), ht)
    _expect("REMP_E_INVALID", rk.Plan, (1, 1), (1, 1), (4, 8, 8, 2, 0, 16), ht)
    bad = rk.HostTables(t.seq_lens, t.offsets, t.ids, 1)                     # ids >= num_blocks
    _expect("REMP_E_RANGE", rk.Plan, (1, 1), (1, 1), shape, bad)
    lens = t.seq_lens.copy()
    lens[0] = -1
    _expect("REMP_E_INVALID", rk.Plan, (1, 1), (1, 1), shape, rk.HostTables(lens, t.offsets, t.ids, t.num_blocks))
    lens = t.seq_lens.copy()
    lens[1] += 40                                                              # row too short
    _expect("REMP_E_INVALID", rk.Plan, (1, 1), (1, 1), shape, rk.HostTables(lens, t.offsets, t.ids, t.num_blocks))
    offs = t.offsets.copy()
    offs[1], offs[2] = offs[2] + 1, offs[1]
    _expect("REMP_E_INVALID", rk.Plan, (1, 1), (1, 1), shape, rk.HostTables(t.seq_lens, offs, t.ids, t.num_blocks))
    # NULL arguments straight through the ABI
    lib = rk.load()
    out = ctypes.c_void_p()
    assert lib.remp_kv_plan(None, None, None, None, ctypes.byref(out)) == -1 and not out.value


def test_plan_accepts_empty_and_zero_length():
    empty = synthkv.tables_from_rows([], [], 0, 16)
    p = rk.Plan((2, 1), (1, 2), (4, 8, 8, 2, 16, 16), rk.HostTables.of(empty))
    assert p.info.total_tokens == 0 and p.info.old_live_blocks == 0
    assert all(q.staging_bytes == 0 for q in p.pairs)
    zl = synthkv.tables_from_rows([0, 0, 5], [[], [], [3]], 4, 16)
    p = rk.Plan((2, 1), (1, 2), (4, 8, 8, 2, 16, 16), rk.HostTables.of(zl))
    assert p.info.total_tokens == 5 and p.info.old_live_blocks == 1


def test_destroy_null_is_noop():
    rk.remp_kv_plan_destroy(None)


# ---------------------------------------------------------------------------
# pack / unpack validation (stand-in device addresses, CPU only)
# ---------------------------------------------------------------------------

class _Fake:
    """Aligned host addresses standing in for device buffers (never dereferenced)."""

    def __init__(self):
        self._keep = []

    def addr(self, nbytes, align=256, offset=0):
        a = np.zeros(nbytes + 2 * align, dtype=np.uint8)
        self._keep.append(a)
        base = a.ctypes.data
        return (base + align - 1) // align * align + offset


def _setup(old=(2, 1), new=(1, 2), L=4, H=8, D=8):
    t = _tables(S=3, n=37, bs=16, N=64)
    free = list(np.random.default_rng(5).permutation(64))
    rows = []
    for n in t.seq_lens:
        k = (int(n) + 15) // 16
        rows.append(free[:k])
        free = free[k:]
    new_t = synthkv.tables_from_rows(t.seq_lens, rows, 64, 16)
    p, _ = _plan(old, new, L, H, D, tables=t)
    f = _Fake()
    per_o, per_n = L // old[1], L // new[1]
    layer_o = [f.addr(64 * 16 * (H // old[0]) * D * 2) for _ in range(2 * per_o)]
    layer_n = [f.addr(64 * 16 * (H // new[0]) * D * 2) for _ in range(2 * per_n)]
    src = rk.PoolArg(layer_o[:per_o], layer_o[per_o:], 64)
    dst = rk.PoolArg(layer_n[:per_n], layer_n[per_n:], 64)
    dev = rk.dev_tables(f.addr(64), f.addr(64), f.addr(1024))
    ws_bytes = p.workspace_bytes
    ws = f.addr(ws_bytes)
    stage = {(q.src, q.dst): (f.addr(q.staging_bytes), q.staging_bytes) for q in p.pairs}
    W_o, W_n = p.info.old_world, p.info.new_world
    out0 = [stage.get((0, q)) for q in range(W_n)]
    in0 = [stage.get((r, 0)) for r in range(W_o)]
    return dict(p=p, t=t, new_t=new_t, f=f, src=src, dst=dst, dev=dev, ws=ws, ws_bytes=ws_bytes,
                out0=out0, in0=in0, L=L, stage=stage)


@cpu_only
def test_pack_validation_errors():
    s = _setup()
    p, L = s["p"], s["L"]
    ok = dict(old_rank=0, src=s["src"], old_dev_tables=s["dev"], staging=rk.buffers(s["out0"]),
              workspace=s["ws"], workspace_bytes=s["ws_bytes"], stream=0, layer_begin=0, layer_end=L, flags=0)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        rk.remp_kv_pack(p.handle, a["old_rank"], a["layer_begin"], a["layer_end"], a["src"], a["old_dev_tables"],
                        a["staging"], a["workspace"], a["workspace_bytes"], a["flags"], a["stream"])

    _expect("REMP_E_RANGE", call, old_rank=2)
    _expect("REMP_E_RANGE", call, old_rank=-1)
    _expect("REMP_E_RANGE", call, layer_begin=3, layer_end=2)
    _expect("REMP_E_RANGE", call, layer_end=L + 1)
    _expect("REMP_E_INVALID", call, src=rk.PoolArg([1] * 3, [1] * 3, 64))          # wrong layer count
    _expect("REMP_E_SIZE", call, src=rk.PoolArg(list(s["src"]._k), list(s["src"]._v), 10))
    _expect("REMP_E_INVALID", call, workspace=0)
    _expect("REMP_E_ALIGN", call, workspace=s["ws"] + 8)
    _expect("REMP_E_SIZE", call, workspace_bytes=s["ws_bytes"] - 1)
    _expect("REMP_E_INVALID", call, old_dev_tables=rk.dev_tables(0, 0, 0))
    bufs = list(s["out0"])
    q = next(i for i, b in enumerate(bufs) if b is not None)
    bufs_null = list(bufs)
    bufs_null[q] = None
    _expect("REMP_E_INVALID", call, staging=rk.buffers(bufs_null))
    bufs_small = list(bufs)
    bufs_small[q] = (bufs[q][0], bufs[q][1] - 2)
    _expect("REMP_E_SIZE", call, staging=rk.buffers(bufs_small))
    bufs_mis = list(bufs)
    bufs_mis[q] = (bufs[q][0] + 1, bufs[q][1])
    _expect("REMP_E_ALIGN", call, staging=rk.buffers(bufs_mis))
    ks = list(s["src"]._k)
    ks[1] = None
    _expect("REMP_E_INVALID", call, src=rk.PoolArg(ks, list(s["src"]._v), 64))
    ks = list(s["src"]._k)
    ks[0] = ks[0] + 1
    _expect("REMP_E_ALIGN", call, src=rk.PoolArg(ks, list(s["src"]._v), 64))
    _expect("REMP_E_INVALID", call, flags=4)
    # with REMP_KV_SKIP_LOCAL the local pair's staging entry may be absent
    local_null = list(s["out0"])
    local_null[0] = None
    _expect("REMP_E_INVALID", call, staging=rk.buffers(local_null), layer_begin=0, layer_end=1)
    lib = rk.load()
    assert lib.remp_kv_pack(None, 0, 0, 1, None, None, None, None, 0, 0, None) == -1
    # an empty window is valid and enqueues nothing
    call(layer_begin=2, layer_end=2)


@cpu_only
def test_unpack_validation_errors():
    s = _setup()
    p, L, nt = s["p"], s["L"], s["new_t"]
    ok = dict(new_rank=0, staging=rk.buffers(s["in0"]), dst=s["dst"], tables=rk.HostTables.of(nt),
              dev=s["dev"], workspace=s["ws"], workspace_bytes=s["ws_bytes"], layer_begin=0, layer_end=L, flags=0)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        rk.remp_kv_unpack(p.handle, a["new_rank"], a["layer_begin"], a["layer_end"], a["staging"], a["dst"],
                          a["tables"], a["dev"], a["workspace"], a["workspace_bytes"], a["flags"], 0)

    _expect("REMP_E_RANGE", call, new_rank=2)
    _expect("REMP_E_INVALID", call, tables=rk.HostTables(nt.seq_lens[:2], nt.offsets[:3], nt.ids, 64))
    lens = nt.seq_lens.copy()
    lens[0] += 1
    _expect("REMP_E_INVALID", call, tables=rk.HostTables(lens, nt.offsets, nt.ids, 64))
    ids = nt.ids.copy()
    ids[0] = 64
    _expect("REMP_E_RANGE", call, tables=rk.HostTables(nt.seq_lens, nt.offsets, ids, 64))
    ids = nt.ids.copy()
    ids[1] = ids[0]
    _expect("REMP_E_INVALID", call, tables=rk.HostTables(nt.seq_lens, nt.offsets, ids, 64))   # duplicate
    _expect("REMP_E_CAPACITY", call, tables=rk.HostTables(nt.seq_lens, nt.offsets, nt.ids, 2))
    big = rk.HostTables(nt.seq_lens, nt.offsets, nt.ids, 65)
    _expect("REMP_E_SIZE", call, tables=big)                                  # dst pool smaller than tables
    _expect("REMP_E_INVALID", call, dev=rk.dev_tables(0, 0, 0))
    _expect("REMP_E_SIZE", call, workspace_bytes=16)
    in0 = list(s["in0"])
    r = next(i for i, b in enumerate(in0) if b is not None)
    in0[r] = (in0[r][0], in0[r][1] // 2)
    _expect("REMP_E_SIZE", call, staging=rk.buffers(in0))
    short = synthkv.tables_from_rows(nt.seq_lens, [nt.row(0)[:-1] if len(nt.row(0)) else [], nt.row(1),
                                                   nt.row(2)], 64, 16)
    if int(nt.seq_lens[0]) > 0:
        _expect("REMP_E_INVALID", call, tables=rk.HostTables.of(short))
    call(layer_begin=0, layer_end=0)
    _expect("REMP_E_INVALID", call, flags=8)


@cpu_only
def test_copy_local_validation_errors():
    s = _setup()
    p, L, nt = s["p"], s["L"], s["new_t"]
    ok = dict(rank=0, src=s["src"], odev=s["dev"], dst=s["dst"], tables=rk.HostTables.of(nt), ndev=s["dev"],
              workspace=s["ws"], workspace_bytes=s["ws_bytes"], layer_begin=0, layer_end=L, flags=0)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        rk.remp_kv_copy_local(p.handle, a["rank"], a["layer_begin"], a["layer_end"], a["src"], a["odev"], a["dst"],
                              a["tables"], a["ndev"], a["workspace"], a["workspace_bytes"], a["flags"], 0)

    _expect("REMP_E_RANGE", call, rank=2)
    _expect("REMP_E_RANGE", call, layer_end=L + 1)
    _expect("REMP_E_INVALID", call, flags=rk.REMP_KV_SKIP_LOCAL)    # pack / unpack only
    _expect("REMP_E_INVALID", call, flags=4)
    _expect("REMP_E_INVALID", call, src=None)
    _expect("REMP_E_INVALID", call, dst=s["src"])                   # wrong layer count for the new topology
    _expect("REMP_E_ALIGN", call, workspace=s["ws"] + 4)
    ids = nt.ids.copy()
    ids[1] = ids[0]
    _expect("REMP_E_INVALID", call, tables=rk.HostTables(nt.seq_lens, nt.offsets, ids, 64))
    _expect("REMP_E_INVALID", call, odev=rk.dev_tables(0, 0, 0))
    # old and new storage of a layer overlapping is refused
    ks = list(s["dst"]._k)
    ks[0] = s["src"]._k[0]
    _expect("REMP_E_INVALID", call, dst=rk.PoolArg(ks, list(s["dst"]._v), 64))
    call(layer_begin=1, layer_end=1)                                 # empty window: nothing to do


def test_one_hip_runtime_in_process():
    """The library binds to the HIP runtime torch loaded (one runtime per process)."""
    rk.load()
    runtimes = rk._lib._mapped_hip_runtimes()
    assert len(runtimes) == 1, runtimes


@cpu_only
def test_layout_validation_errors():
    s = _setup(D=8)          # head_dim 8 * 2 bytes = 16: tile layouts allowed
    p, L = s["p"], s["L"]

    def pack(src):
        rk.remp_kv_pack(p.handle, 0, 0, L, src, s["dev"], rk.buffers(s["out0"]), s["ws"], s["ws_bytes"], 0, 0)

    k, v = list(s["src"]._k), list(s["src"]._v)
    _expect("REMP_E_INVALID", pack, rk.PoolArg(k, v, 64, layout=7))
    s4 = _setup(D=4)         # 8-byte head rows cannot use the tile layouts
    k4, v4 = list(s4["src"]._k), list(s4["src"]._v)
    with pytest.raises(rk.RempError) as ei:
        rk.remp_kv_pack(s4["p"].handle, 0, 0, s4["L"], rk.PoolArg(k4, v4, 64, layout=rk.LAYOUT_HND), s4["dev"],
                        rk.buffers(s4["out0"]), s4["ws"], s4["ws_bytes"], 0, 0)
    assert ei.value.status_name == "REMP_E_UNSUPPORTED"
    # the local copy through head tiles has the same 16-byte head-row requirement
    with pytest.raises(rk.RempError) as ei:
        rk.remp_kv_copy_local(s4["p"].handle, 0, 0, s4["L"], rk.PoolArg(k4, v4, 64, layout=rk.LAYOUT_HND), s4["dev"],
                              s4["dst"], rk.HostTables.of(s4["new_t"]), s4["dev"], s4["ws"], s4["ws_bytes"], 0, 0)
    assert ei.value.status_name == "REMP_E_UNSUPPORTED"


@pytest.mark.parametrize("a,b", [((2, 2, (0, 3, 5)), (1, 1, None)), ((1, 3, (0, 1, 3, 5)), (2, 2, (0, 2, 5))),
                                 ((8, 2, (0, 4, 5)), (4, 5, None)), ((1, 1, None), (2, 5, (0, 1, 2, 3, 4, 5)))])
def test_plan_with_explicit_partition(a, b):
    L, H = 5, 4
    t = _tables()
    p = rk.Plan(a, b, (L, H, 8, 2, 16, 16), rk.HostTables.of(t))
    want = oracle.pair_slices(T(*a), T(*b), L, H)
    got = {(q.src, q.dst): (list(range(q.layer_begin, q.layer_end)),
                            list(range(q.head_begin, q.head_begin + q.head_count))) for q in p.pairs}
    assert got == want


def test_plan_partition_errors():
    t = rk.HostTables.of(_tables())
    shape = (5, 4, 8, 2, 16, 16)
    _expect("REMP_E_UNSUPPORTED", rk.Plan, (1, 2), (1, 1), shape, t)               # 5 % 2 without a partition
    for starts in [(0, 5, 5), (1, 3, 5), (0, 3, 4), (0, 4, 3)]:
        _expect("REMP_E_INVALID", rk.Plan, (1, 2, starts), (1, 1), shape, t)
    _expect("REMP_E_INVALID", rk.Plan, (1, 6), (1, 1), (5, 4, 8, 2, 16, 16), t)    # more stages than layers
