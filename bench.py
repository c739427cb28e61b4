#!/usr/bin/env python3
"""KV-cache migration benchmark on one MI355X.

One step is the whole hot path for one GPU's share of a topology switch:
expand the old block tables and pack everything old rank 0 sends (all its
destinations), then expand the new block tables and unpack everything new
rank 0 receives (from all its sources).  The staging buffers that other old
ranks would send to new rank 0 are produced once, untimed, by packing those
ranks' pools on the same GPU.  All inputs are resident in HBM before timing.

value = algorithmic traffic / step time, with traffic = 2 * (bytes packed +
bytes unpacked): each payload byte is read once and written once per phase.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import statistics
import sys
import time
import types

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E peak, GB/s
PEAK_PCIE_GBS = 64.0   # PCIe Gen5 x16, one direction (32 GT/s x 16 lanes)
PROFILES = os.path.join(ROOT, "profiles")


def counters_path(workload: str) -> str:
    """The committed HBM counter record of a workload's pack and unpack calls."""
    return os.path.join(PROFILES, f"hbm_counters_{workload}.json")
CSRC = os.path.join(ROOT, "paper_2606_18741_amd", "csrc")
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in ("device_util.hpp", "kv_copy.hpp", "kv_device.hpp", "kv_expand.hpp",
                                                  "kv_rows.hpp", "kv_tiles.hpp", "migrate.hip")]


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="gqa70b")
    ap.add_argument("--cpu-sample-layers", type=int, default=24,
                    help="layers per new pipeline stage in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layout", default="nhd", choices=["nhd", "hnd", "rocm"],
                    help="physical layout of both pools (hnd and rocm go through the LDS tile kernel)")
    ap.add_argument("--weight-layers", type=int, default=8,
                    help="decoder layers whose weight shards new rank 0 rebuilds from the host store, for the "
                         "workloads with a model (gqa70b: Llama3-70B, qwen30b: Qwen3-30B-A3B, ds32b: "
                         "DeepSeek-R1-Distill-Qwen-32B; 0: skip the weight-shard measurement)")
    ap.add_argument("--prewarm-gib", type=float, default=200.0,
                    help="GiB of device memory written and released before the workload is allocated (0: none)")
    ap.add_argument("--no-first-touch", action="store_true",
                    help="skip the first-touch measurement (the same steps timed on a workload allocated before "
                         "the prewarm, reported as value_first_touch)")
    ap.add_argument("--seed", type=int, default=None, help="override the workload's seed")
    ap.add_argument("--sigma", type=float, default=None,
                    help="override the lognormal sigma of the workload's sequence lengths")
    ap.add_argument("--stream-windows", default="1,10",
                    help="layers per window for the layer-streaming measurement, comma separated ('' to skip)")
    ap.add_argument("--copy-calibration", type=float, default=0.0, metavar="GIB",
                    help="only run a plain device copy of this many GiB (for counter scaling), then exit")
    ap.add_argument("--library-calibration", type=float, default=0.0, metavar="GIB",
                    help="only run the library's pack on a contiguous pool of this many GiB (one sequence over "
                         "blocks 0..n-1, identity topology: every byte read and written once, in order), then exit")
    ap.add_argument("--counter-pass", action="store_true",
                    help="only build the share and run 3 pack and 3 unpack calls (for rocprofv3 --pmc), then exit")
    ap.add_argument("--summarize-counters", nargs=4, default=None,
                    metavar=("FETCH_CSV", "WRITE_CSV", "CAL_FETCH_CSV", "CAL_WRITE_CSV"),
                    help="write profiles/hbm_counters_<workload>.json from rocprofv3 counter CSVs of a --counter-pass "
                         "run (FETCH_SIZE, WRITE_SIZE) and of a --library-calibration run (same counters), then exit")
    ap.add_argument("--summarize-trace", default=None, metavar="STATS_CSV",
                    help="print a markdown table of a rocprofv3 --stats kernel summary (the library's kernels), "
                         "then exit")
    ap.add_argument("--counter-filter", default=None, metavar="REGEX",
                    help="with --summarize-counters: the --kernel-include-regex the two counter passes ran with "
                         "(recorded in the commands of the record)")
    ap.add_argument("--calibration-gib", type=float, default=4.0,
                    help="size of the --library-calibration pool that the summarized calibration CSVs came from")
    ap.add_argument("--ceiling", type=float, default=0.0, metavar="GIB",
                    help="only run the HBM access-pattern probes (libremp_probe.so) over buffers of this many GiB, "
                         "then exit")
    ap.add_argument("--ceiling-shape", default=None, metavar="THREADS,UNROLL,CHUNKS",
                    help="run the probes at this launch shape only (default: all 48)")
    ap.add_argument("--ceiling-chunks", default="4096,8192",
                    help="chunk sizes of the probes in bytes, comma separated")
    ap.add_argument("--ceiling-window", type=float, default=0.0, metavar="MIB",
                    help="draw the random chunk orders within consecutive windows of this many MiB (0: whole buffer)")
    ap.add_argument("--ceiling-offset", type=int, default=0, metavar="BYTES",
                    help="start every chunk this many bytes (a multiple of 16 below the chunk size) past a chunk "
                         "boundary of the allocation, as staging pieces that start at any token do")
    ap.add_argument("--phased", type=float, default=0.0, metavar="GIB",
                    help="only run the phased-copy probe (a persistent copy whose workgroups wait for each other "
                         "between loads and stores, so the chip reads and writes in separate phases) next to the "
                         "plain contiguous chunk copy, over buffers of this many GiB, then exit")
    return ap.parse_args()


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def source_hash() -> str:
    """Hash of the KV-migration GPU sources (launch code and kernels), comments and white space left
    out, so that only a change of the code itself invalidates counters taken on it."""
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def profiled_call(workload: str, kernel: str):
    """The committed counter record of the workload's `kernel` call ("pack" / "unpack"), if it was taken on
    this kernel source: HBM bytes per call, the kernel it launches and its launches per call; else None."""
    try:
        with open(counters_path(workload)) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("source_hash") != source_hash():
        return None
    return c.get("kernels", {}).get(kernel)


def copy_calibration(gib: float) -> None:
    import torch
    n = int(gib * (1 << 30))
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 5
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"copy_bytes_per_launch_read": n, "copy_bytes_per_launch_write": n, "launches": reps,
                      "ms_per_copy": round(ms, 4), "copy_GBps_read_plus_write": round(2 * n / ms / 1e6, 1)}))


def _calibration_bytes(gib: float) -> int:
    """Bytes the library-calibration pack reads (and writes): K and V of a pool of `gib` GiB, 4 KiB blocks."""
    nblk = int(gib * (1 << 30)) // (2 * 16 * 256)
    return 2 * nblk * 16 * 256


def library_calibration(gib: float) -> int:
    """The library's pack over a contiguous pool: identity topology, one head, one sequence whose table is
    blocks 0..n-1 in order, so the pack kernel reads the whole pool and writes the whole staging buffer once,
    both in address order.  Counter readings of this launch against its known bytes scale FETCH_SIZE and
    WRITE_SIZE for the library's own 16-byte non-temporal accesses."""
    import numpy as np
    import torch

    import paper_2606_18741_amd as rk
    from paper_2606_18741_amd import torch_io as tio

    bs, D = 16, 128
    row = D * 2
    nblk = int(gib * (1 << 30)) // (2 * bs * row)          # K and V pools together hold `gib` GiB
    T = nblk * bs
    lens = np.array([T], np.int32)
    tables = rk.HostTables(lens, np.array([0, nblk], np.int32), np.arange(nblk, dtype=np.int32), nblk)
    plan = rk.Plan((1, 1), (1, 1), (1, 1, D, 2, bs, bs), tables)
    pool = torch.empty((2, nblk, bs, 1, D), dtype=torch.int16, device="cuda")
    pool.fill_(3)
    stage = torch.empty(plan.pairs[0].staging_bytes, dtype=torch.uint8, device="cuda")
    dt = tio.DeviceTables(tables)
    ws = tio.workspace(plan)
    arg = tio.pool_arg([pool], nblk)
    st = tio.staging_args({(0, 0): stage}, 0, 1, as_src=True)
    stream = tio.current_stream()
    reps = 5
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    plan.pack(0, arg, dt.dev, st, ws, ws.numel(), stream)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        plan.pack(0, arg, dt.dev, st, ws, ws.numel(), stream)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    if tio.workspace_flag(ws) != 0 or not torch.equal(stage.view(torch.int16), pool.reshape(-1)):
        print("library calibration: the staging buffer is not the pool", file=sys.stderr)
        return 1
    n = stage.numel()
    print(json.dumps({"kind": "library pack, contiguous", "bytes_read_per_call": n, "bytes_written_per_call": n,
                      "calls": reps + 1, "ms_per_call": round(ms, 4), "GBps_read_plus_write": round(2 * n / ms / 1e6, 1)}))
    return 0


def _counter_rows(path: str):
    """(dispatch id, kernel name, counter name, value) of a rocprofv3 counter-collection CSV, in dispatch order."""
    import csv
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"])))
    rows.sort()
    return rows


def _calls(rows):
    """Split a counter-pass dispatch sequence into library calls: every call starts with expand_scan; a call
    with a sort is an unpack, else a pack.  Returns [(kind, [(kernel, value) of its copy launches])]."""
    calls = []
    for _, name, _, value in rows:
        if "remp::" not in name:
            continue
        if "expand_scan" in name:
            calls.append(["pack", []])
        elif not calls:
            continue
        elif "sort_scan" in name:
            calls[-1][0] = "unpack"
        elif "copy_" in name:
            calls[-1][1].append((name, value))
    return calls


def summarize_counters(args) -> int:
    """profiles/hbm_counters_<workload>.json from a --counter-pass run's FETCH_SIZE and WRITE_SIZE CSVs
    (the last three packs and three unpacks) scaled by a --library-calibration run's readings."""
    import paper_2606_18741_amd as rk
    import synthkv
    fetch_csv, write_csv, cal_fetch_csv, cal_write_csv = args.summarize_counters
    w = synthkv.WORKLOADS[args.workload]
    inp = synthkv.make_inputs(w)
    plan = rk.Plan(w.old_topo, w.new_topo, (w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes,
                                           w.old_block_size, w.new_block_size), rk.HostTables.of(inp.old_tables))
    ro, qn = w.role
    P_pack = sum(p.staging_bytes for p in plan.pairs if p.src == ro)
    P_unpack = sum(p.staging_bytes for p in plan.pairs if p.dst == qn)

    def calib(path, which):
        calls = _calls(_counter_rows(path))
        vals = [sum(v for _, v in c[1]) for c in calls if c[1]]
        return calls[-1][1][0][0], statistics.median(vals)

    # the calibration pool: K and V of args.library_calibration-sized pool, read once and written once
    cal_kernel, cal_fetch = calib(cal_fetch_csv, "fetch")
    _, cal_write = calib(cal_write_csv, "write")
    cal_bytes = _calibration_bytes(args.calibration_gib)
    fetch_scale = cal_bytes / (cal_fetch * 1024)
    write_scale = cal_bytes / (cal_write * 1024)
    flt = f' --kernel-include-regex "{args.counter_filter}"' if args.counter_filter else ""
    out = {"workload": w.name + ": " + w.description, "source_hash": source_hash(),
           "note": "counters of the last 3 pack and 3 unpack calls of a --counter-pass run, summed over the copy "
                   "launches of a call (a call launches once per 8 slices, or per 8 layers for whole rows), "
                   "median over calls, KiB scaled by the library-calibration factors",
           "commands": [f"rocprofv3 --pmc FETCH_SIZE{flt} --output-format csv -d gpurun_out/pmc/{w.name}_fetch -o f -- "
                        f"python bench.py --workload {w.name} --counter-pass",
                        f"rocprofv3 --pmc WRITE_SIZE{flt} --output-format csv -d gpurun_out/pmc/{w.name}_write -o w -- "
                        f"python bench.py --workload {w.name} --counter-pass",
                        f"rocprofv3 --pmc FETCH_SIZE{flt} --output-format csv -d gpurun_out/pmc/cal_fetch -o f -- "
                        f"python bench.py --library-calibration {args.calibration_gib}",
                        f"rocprofv3 --pmc WRITE_SIZE{flt} --output-format csv -d gpurun_out/pmc/cal_write -o w -- "
                        f"python bench.py --library-calibration {args.calibration_gib}",
                        f"python bench.py --workload {w.name} --calibration-gib {args.calibration_gib} "
                        f"--summarize-counters <the four CSVs>"],
           "calibration": {"kernel": cal_kernel, "known_bytes_read": cal_bytes, "known_bytes_written": cal_bytes,
                           "fetch_size_kib": round(cal_fetch, 1), "write_size_kib": round(cal_write, 1),
                           "fetch_scale": round(fetch_scale, 5), "write_scale": round(write_scale, 5)},
           "kernels": {}}
    fetch_calls = _calls(_counter_rows(fetch_csv))
    write_calls = _calls(_counter_rows(write_csv))
    for kind, algo in (("pack", 2 * P_pack), ("unpack", 2 * P_unpack)):
        fc = [c for c in fetch_calls if c[0] == kind and c[1]][-3:]
        wc = [c for c in write_calls if c[0] == kind and c[1]][-3:]
        f_kib = statistics.median(sum(v for _, v in c[1]) for c in fc)
        w_kib = statistics.median(sum(v for _, v in c[1]) for c in wc)
        hbm = f_kib * 1024 * fetch_scale + w_kib * 1024 * write_scale
        out["kernels"][kind] = {"kernel": fc[-1][1][0][0], "launches_per_call": len(fc[-1][1]), "calls": len(fc),
                                "fetch_size_kib_per_call": round(f_kib, 1), "write_size_kib_per_call": round(w_kib, 1),
                                "hbm_bytes_per_call": int(hbm), "algorithmic_bytes_per_call": algo,
                                "hbm_over_algorithmic": round(hbm / algo, 5)}
    with open(counters_path(w.name), "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out["kernels"]))
    return 0


def summarize_trace(path: str) -> int:
    """Markdown table of the library's kernels in a rocprofv3 kernel-stats CSV: calls, average and total time."""
    import csv
    with open(path) as f:
        rows = [r for r in csv.DictReader(f) if "remp::" in r["Name"] or "probe" in r["Name"]]
    print("| kernel | calls | average (ms) | total (ms) |")
    print("|---|---|---|---|")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"].replace("void ", "").replace("remp::", "").split("(")[0]
        print(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | {float(r['TotalDurationNs']) / 1e6:.3f} |")
    return 0


def ceiling(args) -> int:
    """HBM access-pattern probes: 4 and 8 KiB chunks copied (with non-temporal or with device-scope stores),
    read or written in address order or through a random permutation (optionally random only within windows
    of --ceiling-window MiB; every chunk --ceiling-offset bytes past a chunk boundary), each at every launch
    shape (or --ceiling-shape), median of 3 launches; GB/s counts bytes read plus bytes written.  The copy
    patterns are rerun at their best shape into a cleared destination and checked chunk by chunk."""
    gib = args.ceiling
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_18741_amd", "libremp_probe.so"))
    fn = lib.remp_probe_chunks
    fn.restype = ctypes.c_int32
    fn.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_void_p]
    stream = torch.cuda.current_stream()
    shapes = [(t, u, c) for t in (256, 512, 1024) for u in (1, 2, 4, 8) for c in (1, 2, 4, 16)]
    if args.ceiling_shape:
        shapes = [tuple(int(x) for x in args.ceiling_shape.split(","))]
    patterns = [("copy, contiguous", 0, False, False), ("copy, random reads (gather)", 0, True, False),
                ("copy, random writes (scatter)", 0, False, True), ("copy, random reads and writes", 0, True, True),
                ("read only, contiguous", 1, False, False), ("read only, random", 1, True, False),
                ("write only, contiguous", 2, False, False), ("write only, random", 2, False, True),
                ("copy with device-scope stores, contiguous", 3, False, False),
                ("copy with device-scope stores, random reads", 3, True, False)]
    results = []
    for chunk in [int(x) for x in args.ceiling_chunks.split(",")]:
        n = int(gib * (1 << 30)) // chunk
        off = args.ceiling_offset
        if off % 16 or not 0 <= off < chunk:
            raise SystemExit(f"--ceiling-offset {off}: a multiple of 16 below the chunk size {chunk} is needed")
        # the chunks start `off` bytes into the allocations (one chunk more is allocated when off > 0)
        extra = chunk if off else 0
        src_all = torch.randint(0, 256, (n * chunk + extra,), dtype=torch.uint8, device="cuda",
                                generator=torch.Generator(device="cuda").manual_seed(chunk))
        dst_all = torch.empty(n * chunk + extra, dtype=torch.uint8, device="cuda")
        src, dst = src_all[off:off + n * chunk], dst_all[off:off + n * chunk]
        g = torch.Generator(device="cpu").manual_seed(chunk)
        win = max(1, int(args.ceiling_window * (1 << 20)) // chunk) if args.ceiling_window > 0 else n

        def order():
            """A random order of the n chunks, random only within consecutive windows of `win` chunks."""
            parts = [a + torch.randperm(min(win, n - a), generator=g) for a in range(0, n, win)]
            return torch.cat(parts).to(torch.int32).cuda()
        perm_r, perm_w = order(), order()
        sink = torch.empty(1024 * 16, dtype=torch.uint8, device="cuda")
        for name, mode, rr, rw in patterns:
            moved = (2 if mode in (0, 3) else 1) * n * chunk
            best = None
            for (t, u, c) in shapes:
                call = (mode, src.data_ptr(), dst.data_ptr(), sink.data_ptr(), sink.numel(), n, chunk,
                        perm_r.data_ptr() if rr else None, perm_w.data_ptr() if rw else None, t, u, c,
                        stream.cuda_stream)
                if -(-n // c) * t >= (1 << 32):
                    continue                      # more work-items than one dispatch counts
                if fn(*call) != 0:
                    raise RuntimeError(f"probe launch refused: {name} {t}x{u} cpw {c}")
                ts = []
                for _ in range(3):
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    fn(*call)
                    e1.record()
                    e1.synchronize()
                    ts.append(e0.elapsed_time(e1))
                gbps = moved / statistics.median(ts) / 1e6
                if best is None or gbps > best[0]:
                    best = (gbps, t, u, c)
            if mode in (0, 3):
                # the best shape once more into a cleared destination: chunk dst_idx[i] must hold chunk src_idx[i]
                dst.zero_()
                fn(mode, src.data_ptr(), dst.data_ptr(), sink.data_ptr(), sink.numel(), n, chunk,
                   perm_r.data_ptr() if rr else None, perm_w.data_ptr() if rw else None, best[1], best[2], best[3],
                   stream.cuda_stream)
                sv, dv = src.view(n, chunk), dst.view(n, chunk)
                for lo in range(0, n, 1 << 18):
                    hi = min(n, lo + (1 << 18))
                    si = perm_r[lo:hi].long() if rr else torch.arange(lo, hi, device="cuda")
                    di = perm_w[lo:hi].long() if rw else torch.arange(lo, hi, device="cuda")
                    if not torch.equal(dv[di], sv[si]):
                        raise RuntimeError(f"probe copy differs from its source: {chunk} B {name}")
            results.append({"chunk_bytes": chunk, "pattern": name, "GBps": round(best[0], 1),
                            "frac_of_peak": round(best[0] / PEAK_HBM_GBS, 4),
                            "best_shape": {"threads": best[1], "unroll": best[2], "chunks_per_workgroup": best[3]}})
            log(f"ceiling {chunk} B {name}: {best[0]:.1f} GB/s ({best[1]} x {best[2]}, {best[3]} chunks per workgroup)")
        del src, dst, src_all, dst_all, perm_r, perm_w, sink
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "HBM access-pattern ceiling", "unit": "GB/s (read + write)", "buffer_GiB": gib,
                      "random_window_MiB": args.ceiling_window or None, "chunk_offset_bytes": args.ceiling_offset,
                      "shapes_tried": len(shapes),
                      "results": results}))
    return 0


def phased(args) -> int:
    """Phased-copy probe: a contiguous copy by a persistent grid in batches of grid * threads * vecs 16-byte
    vectors, with 0, 1 or 2 grid-wide waits per batch (between the loads and the stores; also after the
    stores), next to the plain contiguous copy of 4 KiB chunks; median of 5 launches, GB/s counts bytes read
    plus bytes written, time-outs are the waits that ended by their 200 us bound.  Each shape's first launch
    is checked byte for byte against the source."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_18741_amd", "libremp_probe.so"))
    chunks = lib.remp_probe_chunks
    chunks.restype = ctypes.c_int32
    chunks.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                       ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                       ctypes.c_int32, ctypes.c_void_p]
    ph = lib.remp_probe_phased
    ph.restype = ctypes.c_int32
    ph.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_int32, ctypes.c_int32, ctypes.c_double, ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p]
    cap = int(args.phased * (1 << 30)) // (1 << 20) * (1 << 20)
    src = torch.randint(0, 256, (cap,), dtype=torch.uint8, device="cuda",
                        generator=torch.Generator(device="cuda").manual_seed(7))
    dst = torch.empty(cap, dtype=torch.uint8, device="cuda")
    sync = torch.zeros(2, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def rate(launch, moved):
        """GB/s of `launch` (moving `moved` bytes), after a first launch into a cleared dst is checked
        byte for byte over the moved range."""
        dst.zero_()
        if launch() != 0:
            raise RuntimeError("probe launch refused")
        if not torch.equal(dst[:moved // 2], src[:moved // 2]):
            raise RuntimeError("probe copy differs from its source")
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            launch()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return moved / statistics.median(ts) / 1e6

    n = cap // 4096
    plain = rate(lambda: chunks(0, src.data_ptr(), dst.data_ptr(), None, 0, n, 4096, None, None, 256, 1, 1, stream),
                 2 * cap)
    log(f"phased probe: plain copy of 4 KiB chunks (256 x 1): {plain:.1f} GB/s")
    results = []
    for t, v in ((256, 8), (512, 8), (1024, 8), (1024, 16)):
        for b in (0, 1, 2):
            res = ctypes.c_int32(0)
            ph(None, None, None, 0, t, v, b, 0, 200.0, ctypes.byref(res), stream)   # refused: asks the resident limit
            for grid in sorted({g for g in (256, res.value) if 0 < g <= res.value}):
                batch = grid * t * v * 16
                nbytes = cap // batch * batch
                if nbytes == 0:
                    continue
                gbps = rate(lambda: ph(src.data_ptr(), dst.data_ptr(), sync.data_ptr(), nbytes, t, v, b, grid, 200.0,
                                       None, stream), 2 * nbytes)
                torch.cuda.synchronize()
                timeouts = int(sync[1].item())
                results.append({"threads": t, "vecs": v, "waits_per_batch": b, "grid": grid,
                                "batch_MiB": batch >> 20, "GBps": round(gbps, 1), "timeouts_last_launch": timeouts})
                log(f"phased probe: {t} x {v}, {b} waits per batch, grid {grid}, batch {batch >> 20} MiB: "
                    f"{gbps:.1f} GB/s ({timeouts} waits timed out)")
    print(json.dumps({"metric": "phased-copy probe", "unit": "GB/s (read + write)", "buffer_GiB": args.phased,
                      "plain_4KiB_chunks_GBps": round(plain, 1), "results": results}))
    return 0


# KV workload -> the decoder whose weights the same switch rebuilds
WEIGHT_MODELS = {"gqa70b": "LLAMA3_70B", "qwen30b": "QWEN3_30B_A3B", "ds32b": "QWEN2_32B"}


def bench_weights(args, rk, synthkv, torch, qn, new_topo, kv_step, kv_ms, dev, spec):
    """Shard rebuild of new rank qn from a page-locked store of `spec` (first args.weight_layers
    layers of its stage plus its non-layer tensors): host-link GB/s alone, then beside the KV step."""
    from synthkv.models import FIRST_STAGE, LAST_STAGE
    tp, pp = new_topo
    stage = qn // tp
    per = spec.num_layers // pp
    window = range(stage * per, stage * per + min(args.weight_layers, per))
    # the store holds what this stage reads: its layers' tensors, plus the embedding on the first
    # stage and the final norm / LM head on the last (the library decides ownership all the same)
    tensors = [t for t in spec.tensors(window)
               if t.layer >= 0 or (t.layer == FIRST_STAGE and stage == 0) or (t.layer == LAST_STAGE and stage == pp - 1)]
    t0 = time.time()
    store = synthkv.models.host_store(spec, pin=True, fill_device=dev, tensors=tensors)
    plan = rk.WeightPlan(new_topo, spec.num_layers, spec.elem_bytes,
                         [(t.layer, [(store[p.name].data_ptr(), p.rows, p.cols, p.split, p.units) for p in t.parts])
                          for t in tensors])
    dst = []
    for i in range(plan.num_tensors):
        r, c = plan.shard_shape(qn, i)
        dst.append(torch.empty(r * c * spec.elem_bytes, dtype=torch.uint8, device=dev) if r else None)
    nbytes = plan.shard_bytes(qn)
    store_bytes = sum(p.rows * p.cols * spec.elem_bytes for t in tensors for p in t.parts)
    log(f"weight store ready: {store_bytes / 1e9:.2f} GB page-locked, shard {nbytes / 1e9:.2f} GB "
        f"({time.time() - t0:.1f}s)")
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()

    def load(flags):
        plan.load(qn, dst, side.cuda_stream, flags=flags)

    def alone(flags, reps=3):
        ts = []
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(side)
            load(flags)
            e1.record(side)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts[1:])

    def together(flags, k):
        """k KV steps on the main stream while one load runs on the side stream, started together."""
        torch.cuda.synchronize()
        s0 = torch.cuda.Event(enable_timing=True)
        em, es = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record(main)
        side.wait_event(s0)
        load(flags)
        es.record(side)
        for _ in range(k):
            kv_step()
        em.record(main)
        torch.cuda.synchronize()
        return s0.elapsed_time(es), s0.elapsed_time(em)

    out = {"model": spec.name, "rank": qn, "topology": f"TP{tp}/PP{pp}",
           "tensors": f"layers {window.start}-{window.stop - 1}" + (" + embedding" if stage == 0 else "")
                      + (" + final norm + LM head" if stage == pp - 1 else ""),
           "store_bytes": store_bytes, "shard_bytes": nbytes, "bound": "host link (PCIe Gen5 x16)",
           "peak_GBps": PEAK_PCIE_GBS}
    for name, flags in (("gather_kernel", 0), ("copy_engine", rk.REMP_W_COPY_ENGINE)):
        ms = alone(flags)
        k = max(1, round(ms / kv_ms))
        load_ms, kv_total = together(flags, k)
        wall = max(load_ms, kv_total)
        out[name] = {"ms": round(ms, 3), "GBps": round(nbytes / ms / 1e6, 1),
                     "frac": round(nbytes / ms / 1e6 / PEAK_PCIE_GBS, 4),
                     "beside_kv": {"kv_steps": k, "kv_ms_alone": round(k * kv_ms, 3),
                                   "load_ms": round(load_ms, 3), "kv_ms": round(kv_total, 3),
                                   "wall_ms": round(wall, 3),
                                   "serial_ms": round(ms + k * kv_ms, 3),
                                   "ideal_ms": round(max(ms, k * kv_ms), 3)}}
        log(f"weights ({name}): {ms:.2f} ms alone, {nbytes / ms / 1e6:.1f} GB/s; beside {k} KV steps: "
            f"load {load_ms:.2f} ms, KV {kv_total:.2f} ms (alone {k * kv_ms:.2f}), wall {wall:.2f} ms")
    del store, dst
    return out


def main() -> int:
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: it plays one rank's share of the migration on one MI355X "
              f"and has no multi-GPU path (asked for --gpus {args.gpus})", file=sys.stderr)
        return 2
    if args.copy_calibration > 0:
        copy_calibration(args.copy_calibration)
        return 0
    if args.ceiling > 0:
        return ceiling(args)
    if args.phased > 0:
        return phased(args)
    if args.library_calibration > 0:
        return library_calibration(args.library_calibration)
    if args.summarize_counters:
        return summarize_counters(args)
    if args.summarize_trace:
        return summarize_trace(args.summarize_trace)

    import numpy as np
    import torch

    import paper_2606_18741_amd as rk
    from paper_2606_18741_amd import torch_io as tio
    import synthkv

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = "cuda:0"
    w = synthkv.WORKLOADS[args.workload]
    if args.seed is not None:
        w = w.replace(seed=args.seed)
    if args.sigma is not None:
        if w.length_law[0] != "lognormal":
            print(f"--sigma applies to lognormal length laws; {w.name} uses {w.length_law[0]}", file=sys.stderr)
            return 2
        w = w.replace(length_law=("lognormal", w.length_law[1], args.sigma, w.length_law[3]))
    if w.role == "all":
        print("bench.py times one rank's share; pick a workload with an (old rank, new rank) role",
              file=sys.stderr)
        return 2
    ro, qn = w.role
    L, H, D = w.num_layers, w.num_kv_heads, w.head_dim
    (tpo, ppo), (tpn, ppn) = w.old_topo, w.new_topo
    layout = {"nhd": rk.LAYOUT_NHD, "hnd": rk.LAYOUT_HND, "rocm": rk.LAYOUT_ROCM_SPLIT}[args.layout]
    if layout != rk.LAYOUT_NHD:
        args.no_cpu_baseline = True        # the oracle's sample reads NHD pools
    inp = synthkv.make_inputs(w)
    shape = (L, H, D, w.elem_bytes, w.old_block_size, w.new_block_size)
    plan = rk.Plan(w.old_topo, w.new_topo, shape, rk.HostTables.of(inp.old_tables))
    W_old, W_new = plan.info.old_world, plan.info.new_world
    pairs_out = [(p.src, p.dst) for p in plan.pairs if p.src == ro]
    pairs_in = [(p.src, p.dst) for p in plan.pairs if p.dst == qn]
    pair_info = {(p.src, p.dst): p for p in plan.pairs}
    P_pack = sum(pair_info[p].staging_bytes for p in pairs_out)
    P_unpack = sum(pair_info[p].staging_bytes for p in pairs_in)
    traffic = 2 * (P_pack + P_unpack)
    log(f"workload {w.name}: T={plan.info.total_tokens} tokens, old blocks {plan.info.old_live_blocks}, "
        f"pack {P_pack / 1e9:.2f} GB, unpack {P_unpack / 1e9:.2f} GB")

    def layers_of(rank, tp, pp):
        per = L // pp
        return range((rank // tp) * per, (rank // tp + 1) * per)

    dt = synthkv.torch_dtype_for(w.elem_bytes)
    nd = synthkv.numpy_dtype_for(w.elem_bytes)

    def alloc_layer(tables, tp):
        h_loc = H // tp if tp <= H else 1          # with more tensor ranks than KV heads: one replica each
        return torch.empty((2, tables.num_blocks, tables.block_size, h_loc, D), dtype=dt, device=dev)

    keep_layers = set()
    if not args.no_cpu_baseline:
        per_new = L // ppn
        k = max(1, min(args.cpu_sample_layers, per_new))
        keep_layers = {s * per_new + i for s in range(ppn) for i in range(k)}

    def build(keep_host: bool):
        """Allocate and fill the share: old rank ro's pools, new rank qn's pools, every staging buffer ro
        fills or qn reads, the workspace; the staging other old ranks send to qn is packed once, untimed
        (each foreign source packs its whole share, so every pack launch in a profile has one shape).
        keep_host: keep host copies of the foreign sources' sampled layers for the oracle."""
        t0 = time.time()
        sh = types.SimpleNamespace()
        sh.src_layers = {}
        for l in layers_of(ro, tpo, ppo):
            t = alloc_layer(inp.old_tables, tpo)
            for kv in range(2):
                synthkv.fill_pool_layer_(t[kv], w.seed, ro, l, kv)
            sh.src_layers[l] = t
        # the same bytes serve any layout: the migration is a permutation of them
        sh.src_arg = tio.pool_arg([sh.src_layers[l] for l in layers_of(ro, tpo, ppo)], inp.old_tables.num_blocks,
                                  layout)
        sh.dst_layers = {l: alloc_layer(inp.new_tables, tpn) for l in layers_of(qn, tpn, ppn)}
        sh.dst_arg = tio.pool_arg([sh.dst_layers[l] for l in layers_of(qn, tpn, ppn)], inp.new_tables.num_blocks,
                                  layout)
        sh.dto = tio.DeviceTables(rk.HostTables.of(inp.old_tables), dev)
        sh.dtn = tio.DeviceTables(rk.HostTables.of(inp.new_tables), dev)
        sh.staging = tio.alloc_staging(plan, sorted(set(pairs_out) | set(pairs_in)), dev)
        sh.ws = tio.workspace(plan, dev)
        sh.stream = tio.current_stream()
        torch.cuda.synchronize()
        log(f"pools and staging allocated and filled ({time.time() - t0:.1f}s)")
        sh.foreign_host = {}
        for (r, q) in pairs_in:
            if r == ro:
                continue
            tmp = {}
            for l in layers_of(r, tpo, ppo):
                t = alloc_layer(inp.old_tables, tpo)
                for kv in range(2):
                    synthkv.fill_pool_layer_(t[kv], w.seed, r, l, kv)
                tmp[l] = t
                if keep_host and l in keep_layers and pair_info[(r, q)].layer_begin <= l < pair_info[(r, q)].layer_end:
                    sh.foreign_host[(r, l)] = t.cpu().numpy().view(nd)
            arg = tio.pool_arg([tmp[l] for l in layers_of(r, tpo, ppo)], inp.old_tables.num_blocks, layout)
            extra = tio.alloc_staging(plan, [pp for pp in pair_info if pp[0] == r and pp != (r, q)], dev)
            bufs = dict(extra)
            bufs[(r, q)] = sh.staging[(r, q)]
            plan.pack(r, arg, sh.dto.dev, tio.staging_args(bufs, r, W_new, as_src=True), sh.ws, sh.ws.numel(),
                      sh.stream)
            torch.cuda.synchronize()
            log(f"staging of old rank {r} for new rank {q} packed ({time.time() - t0:.1f}s)")
            if tio.workspace_flag(sh.ws) != 0:
                raise RuntimeError("device tables disagree with host tables")
            del tmp, arg, extra, bufs
            torch.cuda.empty_cache()
        sh.st_out = tio.staging_args(sh.staging, ro, W_new, as_src=True)
        sh.st_in = tio.staging_args(sh.staging, qn, W_old, as_src=False)
        log(f"share built: pools, staging and foreign staging ready ({time.time() - t0:.1f}s)")
        return sh

    def step(sh, ev=None):
        if ev is not None:
            rk.remp_kv_set_trace_events(ev[0].cuda_event, ev[1].cuda_event)
        plan.pack(ro, sh.src_arg, sh.dto.dev, sh.st_out, sh.ws, sh.ws.numel(), sh.stream)
        if ev is not None:
            rk.remp_kv_set_trace_events(ev[2].cuda_event, ev[3].cuda_event)
        plan.unpack(qn, sh.st_in, sh.dst_arg, sh.dtn.host, sh.dtn.dev, sh.ws, sh.ws.numel(), sh.stream)
        if ev is not None:
            rk.remp_kv_set_trace_events(None, None)

    def timed(sh):
        """args.warmup untimed steps, then args.steps steps between two events, with per-call events."""
        for _ in range(args.warmup):
            step(sh)
        torch.cuda.synchronize()
        if tio.workspace_flag(sh.ws) != 0:
            raise RuntimeError("device tables disagree with host tables")
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        for e4 in evs:           # torch creates the HIP event on first record; the library re-records it
            for e in e4:
                e.record()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for i in range(args.steps):
            step(sh, evs[i])
        stop.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop) / max(args.steps, 1)
        return ms, [e[0].elapsed_time(e[1]) for e in evs], [e[2].elapsed_time(e[3]) for e in evs]

    if args.counter_pass:
        # the calls rocprofv3 --pmc reads: the share's pack and unpack, three times each
        sh = build(keep_host=False)
        for _ in range(3):
            step(sh)
        torch.cuda.synchronize()
        if tio.workspace_flag(sh.ws) != 0:
            raise RuntimeError("device tables disagree with host tables")
        log("counter pass: 3 pack and 3 unpack calls done")
        return 0
    first_touch = None
    if not args.no_first_touch:
        # the same steps on a share allocated before any prewarm of device memory
        sh = build(keep_host=False)
        ft_ms, _, _ = timed(sh)
        first_touch = {"value": round(traffic / (ft_ms / 1e3) / 1e9, 1), "ms_per_step": round(ft_ms, 4)}
        log(f"first touch: {ft_ms:.3f} ms/step, {first_touch['value']} GB/s")
        del sh
        torch.cuda.empty_cache()
    if args.prewarm_gib > 0:
        # First use of device memory that no process has used since the machine started is measurably
        # slower for the scattered unpack writes (MI355X: 5.58-5.66 TB/s in a machine's first benchmark
        # process against 5.76-5.84 TB/s in later ones); a serving engine's KV pool is long resident.
        # Write and release most of the memory once before allocating the workload.
        free, _ = torch.cuda.mem_get_info()
        n = min(int(args.prewarm_gib * (1 << 30)), int(free * 0.9))
        scratch = torch.empty(n, dtype=torch.uint8, device=dev)
        scratch.fill_(0)
        torch.cuda.synchronize()
        del scratch
        torch.cuda.empty_cache()
    sh = build(keep_host=not args.no_cpu_baseline)
    src_layers, dst_layers, staging, ws, stream = sh.src_layers, sh.dst_layers, sh.staging, sh.ws, sh.stream
    src_arg, dst_arg, dto, dtn = sh.src_arg, sh.dst_arg, sh.dto, sh.dtn
    ms_per_step, pack_ms, unpack_ms = timed(sh)
    value = traffic / (ms_per_step / 1e3) / 1e9
    log(f"{args.steps} steps: {ms_per_step:.3f} ms/step, pack kernel {statistics.mean(pack_ms):.3f} ms, "
        f"unpack kernel {statistics.mean(unpack_ms):.3f} ms, {value:.1f} GB/s")
    # what the timed steps wrote in the oracle's sample layers, copied out before anything else runs
    sample = sorted(keep_layers)
    got_dst, got_stage = {}, {}
    if sample:
        got_dst = {l: dst_layers[l].cpu() for l in sample if l in dst_layers}
        for key in sorted(set(pairs_out) | set(pairs_in)):
            _, offs = plan.query(*key)
            got_stage[key] = {l: staging[key][int(offs[l]):int(offs[l + 1])].cpu() for l in sample
                              if pair_info[key].layer_begin <= l < pair_info[key].layer_end}

    # --- the same share with the local fast path (slices old rank ro keeps as new
    # rank qn go pool to pool; the rest through staging), timed the same way
    local = None
    if ro == qn and (ro, qn) in pair_info:
        P_local = pair_info[(ro, qn)].staging_bytes
        st_out_r = tio.staging_args({k: v for k, v in staging.items() if k[0] == ro and k[1] != ro}, ro, W_new, True)
        st_in_r = tio.staging_args({k: v for k, v in staging.items() if k[1] == qn and k[0] != qn}, qn, W_old, False)

        def step_local():
            plan.pack(ro, src_arg, dto.dev, st_out_r, ws, ws.numel(), stream, flags=rk.REMP_KV_SKIP_LOCAL)
            plan.copy_local(ro, src_arg, dto.dev, dst_arg, dtn.host, dtn.dev, ws, ws.numel(), stream)
            plan.unpack(qn, st_in_r, dst_arg, dtn.host, dtn.dev, ws, ws.numel(), stream, flags=rk.REMP_KV_SKIP_LOCAL)

        for _ in range(args.warmup):
            step_local()
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record()
        for _ in range(args.steps):
            step_local()
        a1.record()
        torch.cuda.synchronize()
        if tio.workspace_flag(ws) != 0:
            raise RuntimeError("device tables disagree with host tables")
        ms_local = a0.elapsed_time(a1) / max(args.steps, 1)
        moved = traffic - 2 * P_local
        local = {"ms_per_step": round(ms_local, 4), "speedup_vs_staged": round(ms_per_step / ms_local, 3),
                 "hbm_traffic_bytes": moved, "hbm_GBps": round(moved / (ms_local / 1e3) / 1e9, 1),
                 "local_bytes": P_local}
        log(f"local fast path: {ms_local:.3f} ms/step ({ms_per_step / ms_local:.2f}x), "
            f"{local['hbm_GBps']} GB/s of HBM traffic")

    # --- layer streaming: the same share as one pack and one unpack call per window of layers ---
    streaming = []
    for per in [int(x) for x in args.stream_windows.split(",") if x.strip()]:
        if per < 1 or per >= L:
            continue
        wins = [(a, min(L, a + per)) for a in range(0, L, per)]
        wargs = [(tio.staging_args(staging, ro, W_new, True, plan, x), tio.staging_args(staging, qn, W_old, False,
                                                                                       plan, x), x) for x in wins]

        def step_windows(reuse):
            # with reuse, the step's first pack and first unpack expand the tables, the other windows
            # take the descriptors they left in the workspace
            for i, (so, si, (a, b)) in enumerate(wargs):
                fl = rk.REMP_KV_REUSE_DESCRIPTORS if (reuse and i) else 0
                plan.pack(ro, src_arg, dto.dev, so, ws, ws.numel(), stream, a, b, flags=fl)
                plan.unpack(qn, si, dst_arg, dtn.host, dtn.dev, ws, ws.numel(), stream, a, b, flags=fl)

        row = {"layers_per_window": per, "windows": len(wins)}
        for reuse in (False, True):
            for _ in range(args.warmup):
                step_windows(reuse)
            torch.cuda.synchronize()
            b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            b0.record()
            for _ in range(args.steps):
                step_windows(reuse)
            b1.record()
            torch.cuda.synchronize()
            if tio.workspace_flag(ws) != 0:
                raise RuntimeError(f"workspace flag {tio.workspace_flag(ws)} after layer streaming")
            ms_w = b0.elapsed_time(b1) / max(args.steps, 1)
            key = "reuse_descriptors" if reuse else "expand_every_call"
            row[key] = {"ms_per_step": round(ms_w, 4), "GBps": round(traffic / (ms_w / 1e3) / 1e9, 1)}
            log(f"layer streaming, {per} layers per window, {key.replace('_', ' ')}: {ms_w:.3f} ms/step")
        streaming.append(row)

    weights = None
    spec = WEIGHT_MODELS.get(w.name)
    if args.weight_layers > 0 and spec is not None:
        weights = bench_weights(args, rk, synthkv, torch, qn, w.new_topo, lambda: step(sh), ms_per_step, dev,
                                getattr(synthkv, spec))

    pack_avg, unpack_avg = statistics.mean(pack_ms), statistics.mean(unpack_ms)
    if pack_avg >= unpack_avg:
        dom, dom_ms, dom_bytes = "pack", pack_avg, 2 * P_pack
    else:
        dom, dom_ms, dom_bytes = "unpack", unpack_avg, 2 * P_unpack
    achieved = dom_bytes / (dom_ms / 1e3) / 1e9
    prof = profiled_call(w.name, dom)
    kname = prof["kernel"].replace("void remp::", "").split("<")[0] if prof else "copy kernel"
    roofline = {
        "bound": "hbm",
        "kernel": f"{kname} ({dom})",
        "achieved": round(achieved, 1),
        "peak": PEAK_HBM_GBS,
        "unit": "GB/s",
        "frac": round(achieved / PEAK_HBM_GBS, 4),
        "traffic": prof["hbm_bytes_per_call"] if prof else None,
        # a call launches its kernel once per 8 slices (or 8 layers for whole rows); bytes and time are
        # per call (HIP events around all of its launches, gaps included)
        "algorithmic_bytes_per_call": dom_bytes,
        "avg_call_ms": round(dom_ms, 4),
        "launches_per_call": prof["launches_per_call"] if prof else None,
    }

    # --- CPU baseline: the oracle on a bounded sample of the same workload, and the timed output checked
    # against it ----
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle
        old_h = {ro: {l: src_layers[l].cpu().numpy().view(nd) for l in sample if l in src_layers}}
        for (r, l), a in sh.foreign_host.items():
            old_h.setdefault(r, {})[l] = a
        # pre-filled with what the GPU left there, so the comparison below checks the rows the oracle writes
        # (every live row of the sample layers); dead rows are compared by the test suite
        new_h = {qn: {l: got_dst[l].numpy().view(nd).copy() for l in got_dst}}
        want = sorted(set(pairs_out) | set(pairs_in))
        log(f"oracle on layers {sample} ...")
        t1 = time.perf_counter()
        ref = oracle.reshard(old_h, new_h, oracle.Topology(tpo, ppo), oracle.Topology(tpn, ppn), L, H,
                             inp.old_tables, inp.new_tables, layers=sample, pairs=want)
        cpu_s = time.perf_counter() - t1
        moved = 0
        for key in want:
            p = pair_info[key]
            n_l = len([l for l in sample if p.layer_begin <= l < p.layer_end])
            moved += 2 * n_l * p.slice_bytes * (2 if (key in pairs_out and key in pairs_in) else 1)
        cpu_value = moved / cpu_s / 1e9
        cpu = {"value": round(cpu_value, 3), "unit": "GB/s", "cores": 1, "kind": "oracle", "cpu_model": cpu_model(),
               "seconds": round(cpu_s, 2),
               "sample": f"layers {sample} of the same workload and role: pack slices of old rank {ro} "
                         f"and unpack slices of new rank {qn} in those layers ({moved / 1e9:.2f} GB of "
                         f"traffic by the same definition); NumPy, one thread"}
        log(f"oracle: {cpu_s:.1f}s, {cpu_value:.2f} GB/s")
        # the same oracle and sample, one layer per task on a thread pool the size of this
        # process's CPU share (NumPy's copies release the interpreter lock)
        import concurrent.futures
        threads = len(os.sched_getaffinity(0))
        t1 = time.perf_counter()
        with concurrent.futures.ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda l: oracle.reshard(old_h, new_h, oracle.Topology(tpo, ppo), oracle.Topology(tpn, ppn),
                                                 L, H, inp.old_tables, inp.new_tables, layers=[l], pairs=want)
                        and None, sample))
        par_s = time.perf_counter() - t1
        cpu["parallel"] = {"value": round(moved / par_s / 1e9, 3), "unit": "GB/s", "cores": threads,
                           "seconds": round(par_s, 2), "how": "one layer per task, ThreadPoolExecutor"}
        log(f"oracle on {threads} threads: {par_s:.1f}s, {moved / par_s / 1e9:.2f} GB/s")

        bad, checked = [], 0
        for key, per_layer in got_stage.items():
            for l, g in per_layer.items():
                e = np.ascontiguousarray(ref[key][l]).reshape(-1).view(np.uint8)
                if not torch.equal(g, torch.from_numpy(e)):
                    bad.append(f"staging {key} layer {l}")
                checked += g.numel()
        for l, g in got_dst.items():
            e = new_h[qn][l]
            if not torch.equal(g.view(-1).view(torch.uint8),
                               torch.from_numpy(np.ascontiguousarray(e).reshape(-1).view(np.uint8))):
                bad.append(f"new pool layer {l}")
            checked += g.numel() * g.element_size()
        parity = {"ok": not bad, "against": "oracle", "layers": sample, "compared_bytes": checked,
                  "mismatches": bad[:20],
                  "what": f"every staging byte of the pairs old rank {ro} fills and new rank {qn} reads, and every "
                          f"live row of new rank {qn}'s pool, in the sample layers, as the timed steps left them"}
        log(f"parity against the oracle: {'ok' if not bad else 'MISMATCH ' + ', '.join(bad[:5])} "
            f"({checked / 1e9:.2f} GB compared)")

    out = {
        "metric": "KV migration GB/s (pack+unpack) and % of MI355X HBM peak, 70B GQA share",
        "value": round(value, 1),
        "unit": "GB/s",
        "pct_of_hbm_peak": round(100 * value / PEAK_HBM_GBS, 2),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u16",
        "data": "synthetic",
        "config": {
            "workload": w.name + ": " + w.description,
            "role": f"old rank {ro} packs for all destinations, new rank {qn} unpacks from all sources",
            "pool_layout": args.layout,
            "total_tokens": plan.info.total_tokens,
            "pack_bytes": P_pack,
            "unpack_bytes": P_unpack,
            "traffic_bytes": traffic,
            "payload_GBps": round((P_pack + P_unpack) / (ms_per_step / 1e3) / 1e9, 1),
            "metadata_bytes": plan.workspace_bytes,
            "pack_kernel_ms": round(pack_avg, 4),
            "unpack_kernel_ms": round(unpack_avg, 4),
        },
        "parity": parity,
        "value_first_touch": first_touch["value"] if first_touch else None,
        "first_touch": first_touch,
        "roofline": roofline,
        "local_fast_path": local,
        "layer_streaming": streaming,
        "weights": weights,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    if parity is not None and not parity["ok"]:
        print("bench.py: the timed output differs from the oracle", file=sys.stderr)
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main())
