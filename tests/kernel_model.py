"""CPU model of the KV-migration kernels, for bounds and write-count checks.

Test infrastructure.  It restates, in NumPy, what libremp_kv.so's launch code
decides (vector width, units per workgroup, grid shape, slices per launch, the
choice between the row, whole-row and head-tile kernels) and the per-lane index
arithmetic of every kernel (expand_scan / expand_emit, the descriptor bucket
sort, copy_slices, copy_rows, copy_tiles, copy_local, copy_local_tiles), over a
simulated address space in which every buffer is a region of its own:

* every load and store is checked against the region it must stay inside
  (device tables, workspace areas, pools, staging) and the LDS array it uses;
* every store is counted, so a byte written twice (two lanes racing, or a row
  copied twice) is caught, and the caller can check which bytes were written;
* 32-bit index arithmetic is checked for wrap-around.

A migration run through the model yields real bytes, which the tests compare
with the oracle.  The model reads the plan's pairs through the package's host
planner (no GPU involved) and never runs a kernel.

Regions can be "virtual" (a size and no bytes): then only the bounds of the
accesses are checked, which lets the tests walk sampled workgroups of the
full-size launches without holding their pools.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# launch constants, as in kv_device.hpp / kv_rows.hpp / kv_tiles.hpp / kv_copy.hpp
MAX_ITEMS = 8
MAX_UNITS_PER_WG = 128
SMALL_UNIT_BYTES = 16 * 1024
SMALL_WG_BYTES = 4 * 1024
LARGE_WG_BYTES = 64 * 1024
LOCAL_SMALL_WG_BYTES = 16 * 1024
LOCAL_LARGE_WG_BYTES = 32 * 1024
MAX_WG_VECTORS = 1 << 31
MAX_LOCAL_ROWS = 1024
MAX_LOCAL_ITEMS = 8
MAX_MERGE_SEGS = 4
MAX_MERGE_GROUPS = 8
UNPACK_ROWS_MIN, UNPACK_ROWS_MAX = 256, 0xFFFFFFFF
PACK_ROWS_MIN, PACK_ROWS_MAX = 256, 256
TILE_THREADS = 256
TILE_LDS_BYTES = 32 * 1024
TILE_WG_BYTES = 16 * 1024
DESCS_PER_BUCKET = 4
NHD, HND, ROCM = 0, 1, 2
INT32_MAX = 2 ** 31 - 1
EMIT_CHUNK = 1 << 23          # expand_emit lanes modelled at once

# (threads, loads per lane, XCD cell order) of each launch kind
PACK_SMALL = (64, 4, False)
PACK_PARTIAL = (256, 1, False)      # small-unit pack whose slices take part of each row
UNPACK_TINY = (64, 4, False)        # small-unit unpack moving at most 4 KiB per workgroup
UNPACK_TINY_WG_BYTES = 4 * 1024
UNPACK_SMALL = (128, 4, False)
LARGE = (1024, 2, True)
ROWS_SMALL = (256, 2, False)
ROWS_LARGE = (1024, 2, True)
LOCAL_SMALL = (256, 2, False)
LOCAL_LARGE = (512, 4, True)


class ModelError(AssertionError):
    pass


# ---------------------------------------------------------------------------
# integer helpers with the kernels' semantics
# ---------------------------------------------------------------------------

def make_fastdiv(d: int) -> Tuple[int, int]:
    """Granlund-Montgomery magic number and shift for division by d (as the library computes them)."""
    l = 0
    while (1 << l) < d:
        l += 1
    m = ((1 << 32) * ((1 << l) - d)) // d + 1
    if not 0 <= m < (1 << 32):
        raise ModelError(f"fast division magic out of 32 bits for d={d}")
    return m, l


def fast_div(n: np.ndarray, magic: int, shift: int) -> np.ndarray:
    """(mulhi(n, magic) + n) >> shift in 33 bits, for uint32 n."""
    n = np.asarray(n, dtype=np.uint64)
    if (n >= (1 << 32)).any():
        raise ModelError("fast division of a numerator beyond 32 bits")
    t = (n * np.uint64(magic)) >> np.uint64(32)
    return ((t + n) >> np.uint64(shift)).astype(np.int64)


def div_checked(n: np.ndarray, d: int) -> Tuple[np.ndarray, np.ndarray]:
    """Quotient and remainder through the kernels' fast division, checked against exact division."""
    m, s = make_fastdiv(d)
    q = fast_div(n, m, s)
    if (q != np.asarray(n, dtype=np.int64) // d).any():
        raise ModelError(f"fast division by {d} is wrong for some numerator")
    return q, np.asarray(n, dtype=np.int64) - q * d


def cdiv_trunc(a: np.ndarray, b: int) -> np.ndarray:
    """C integer division (truncation toward zero)."""
    a = np.asarray(a, dtype=np.int64)
    return np.sign(a) * (np.abs(a) // b)


def check_grid(gx: int, gy: int, threads: int, what: str) -> None:
    """The launch code's refusal of grids whose work-items or workgroups overflow 32 bits."""
    if gx * threads >= (1 << 32) or gx * gy >= (1 << 32):
        raise ModelError(f"unsupported: {what}: too many workgroups for one launch")


def lowest_bit(x: int) -> int:
    return x & -x


def grid_cells(gx: int, gy: int, xcd: bool) -> Tuple[np.ndarray, np.ndarray]:
    """(cx, cy) of every workgroup in linear dispatch order (blockIdx.y * gx + blockIdx.x), as grid_cell<XCD>."""
    lin = np.arange(gx * gy, dtype=np.int64)
    if not xcd:
        return lin % gx, lin // gx
    total = gx * gy
    q, r = total // 8, total % 8
    k = lin % 8
    cell = k * q + np.minimum(k, r) + lin // 8
    return cell % gx, cell // gx


# ---------------------------------------------------------------------------
# simulated memory
# ---------------------------------------------------------------------------

@dataclass
class Region:
    base: int
    size: int
    name: str
    data: Optional[np.ndarray]        # uint8 view, or None for a virtual region
    writes: Optional[np.ndarray]      # per-byte store counts (None for virtual)


class Mem:
    """Address space of separate regions; loads and stores are bounds-checked and stores counted."""

    GAP = 1 << 24

    def __init__(self):
        self.regions: List[Region] = []
        self.next = 1 << 40
        self._bases = np.zeros(0, np.int64)

    def add(self, name: str, data: Optional[np.ndarray] = None, size: Optional[int] = None,
            align: int = 256) -> int:
        if data is not None:
            data = np.ascontiguousarray(data).reshape(-1).view(np.uint8)
            size = data.size
        base = (self.next + align - 1) // align * align
        self.next = base + max(int(size), 1) + self.GAP
        self.regions.append(Region(base, int(size), name, data,
                                   np.zeros(int(size), np.uint8) if data is not None else None))
        self._bases = np.array([r.base for r in self.regions], np.int64)
        self._sizes = np.array([r.size for r in self.regions], np.int64)
        self._names = {r.name: r for r in self.regions}
        return base

    def region(self, name: str) -> Region:
        return self._names[name]

    def _locate(self, addrs: np.ndarray, n: int, what: str):
        addrs = np.asarray(addrs, dtype=np.int64)
        k = np.searchsorted(self._bases, addrs, side="right") - 1
        if (k < 0).any():
            raise ModelError(f"{what}: address below every buffer")
        off = addrs - self._bases[k]
        bad = off + n > self._sizes[k]
        if bad.any():
            i = int(np.nonzero(bad)[0][0])
            reg = self.regions[int(k[i])]
            raise ModelError(f"{what}: {n}-byte access at offset {int(off[i])} of {reg.name} "
                             f"({reg.size} bytes)")
        return k, off

    # accesses of one call are modelled in chunks of this many lanes, to bound the temporaries
    CHUNK = 1 << 20

    def load(self, addrs, n: int, what: str) -> np.ndarray:
        addrs = np.asarray(addrs, dtype=np.int64).reshape(-1)
        out = np.zeros((addrs.size, n), np.uint8)
        for a in range(0, addrs.size, self.CHUNK):
            part = addrs[a:a + self.CHUNK]
            k, off = self._locate(part, n, what)
            for ri in np.unique(k):
                m = k == ri
                reg = self.regions[int(ri)]
                if reg.data is not None:
                    out[a:a + self.CHUNK][m] = reg.data[off[m][:, None] + np.arange(n)]
        return out

    def store(self, addrs, vals: np.ndarray, what: str) -> None:
        """Stores of one call; a byte stored twice (by two lanes, or by this call and an earlier one since
        the last reset_writes) is an error."""
        addrs = np.asarray(addrs, dtype=np.int64).reshape(-1)
        for a in range(0, addrs.size, self.CHUNK):
            self._store(addrs[a:a + self.CHUNK], vals[a:a + self.CHUNK], what)

    def _store(self, addrs: np.ndarray, vals: np.ndarray, what: str) -> None:
        if addrs.size == 0:
            return
        n = vals.shape[1]
        k, off = self._locate(addrs, n, what)
        for ri in np.unique(k):
            m = k == ri
            reg = self.regions[int(ri)]
            if reg.data is None:
                continue
            o = off[m]
            # stores of one call start at distinct addresses aligned to a power of two >= their width, so
            # their bytes are distinct exactly when their start addresses are
            if np.unique(o).size != o.size:
                raise ModelError(f"{what}: two lanes store to the same address of {reg.name}")
            w = 1 << (n - 1).bit_length()
            if (o % min(w, 16)).any():
                raise ModelError(f"{what}: a {n}-byte store is not aligned to its width")
            idx = (o[:, None] + np.arange(n)).reshape(-1)
            reg.writes[idx] += 1
            if reg.writes[idx].max() > 1:
                raise ModelError(f"{what}: a byte of {reg.name} is written twice")
            reg.data[idx] = vals[m].reshape(-1)

    def load_i32(self, addr: int, index, what: str) -> np.ndarray:
        index = np.asarray(index, dtype=np.int64)
        raw = self.load(addr + 4 * index.reshape(-1), 4, what)
        return raw.view(np.int32).reshape(index.shape).astype(np.int64)

    def store_i32(self, addr: int, index, values, what: str) -> None:
        index = np.asarray(index, dtype=np.int64).reshape(-1)
        v = np.asarray(values, dtype=np.int64).reshape(-1).astype(np.int32).view(np.uint8).reshape(-1, 4)
        self.store(addr + 4 * index, v, what)

    def reset_writes(self) -> None:
        for r in self.regions:
            if r.writes is not None:
                r.writes[:] = 0


# ---------------------------------------------------------------------------
# expansion and sort
# ---------------------------------------------------------------------------

@dataclass
class Tables:
    """Device tables as the kernels see them: addresses of seq_lens [S], row_offsets [S+1], block_ids [nnz]."""
    lens: int
    offs: int
    ids: int


@dataclass
class Expanded:
    desc: np.ndarray          # [n, 4] (block, tok, n, seq)
    tok_off: np.ndarray       # [S+1]
    blk_off: np.ndarray       # [S+1]
    flag: int


def expand(mem: Mem, tables: Tables, S: int, bs: int, nnz: int, num_blocks: int, total_tokens: int,
           n_desc: int, scan_addr: int, desc_addr: int, bucket_addr: Optional[int] = None,
           nb: int = 0) -> Expanded:
    """expand_scan (one workgroup) then expand_emit (one lane per live block): writes the token and
    block offsets to scan_addr, the descriptors to desc_addr and counts the sort buckets."""
    flag = 0
    if bucket_addr is not None and nb:
        mem.store_i32(bucket_addr, np.arange(nb), np.zeros(nb), "expand_scan: bucket clear")
    lens = mem.load_i32(tables.lens, np.arange(S), "expand_scan: seq_lens") if S else np.zeros(0, np.int64)
    if (lens < 0).any():
        flag = 1
    n = np.maximum(lens, 0)
    nblk = (n + bs - 1) // bs
    tok = np.concatenate([[0], np.cumsum(n)])
    blk = np.concatenate([[0], np.cumsum(nblk)])
    if (tok[:-1] > INT32_MAX).any() or (blk[:-1] > INT32_MAX).any():
        flag = 1
    tok_off = np.minimum(tok, INT32_MAX)
    blk_off = np.minimum(blk, INT32_MAX)
    mem.store_i32(scan_addr, np.arange(S + 1), tok_off, "expand_scan: token offsets")
    mem.store_i32(scan_addr + 4 * (S + 1), np.arange(S + 1), blk_off, "expand_scan: block offsets")

    # (block, tok, n, seq) per descriptor; every field of a descriptor the kernel emits fits int32
    desc = np.zeros((n_desc, 4), np.int32)
    for c0 in range(0, n_desc, EMIT_CHUNK):     # lanes in chunks, to bound the temporaries
        b = np.arange(c0, min(n_desc, c0 + EMIT_CHUNK), dtype=np.int64)
        # last s in [0, S] with blk_off[s] <= b (binary search over the block offsets the scan wrote)
        lo = np.searchsorted(blk_off, b, side="right") - 1
        lo = np.clip(lo, 0, S)
        mem.load_i32(scan_addr + 4 * (S + 1), np.unique(np.clip(lo, 0, S)), "expand_emit: block offsets")
        ok = lo < S
        s = np.where(ok, lo, 0)
        j = b - blk_off[s]
        nn = np.zeros(b.size, np.int64)
        r = np.zeros(b.size, np.int64)
        if ok.any():
            nn[ok] = mem.load_i32(tables.lens, s[ok], "expand_emit: seq_lens")
            r[ok] = mem.load_i32(tables.offs, s[ok], "expand_emit: row_offsets") + j[ok]
        ok &= (r >= 0) & (r < nnz)
        ids = np.zeros(b.size, np.int64)
        if ok.any():
            ids[ok] = mem.load_i32(tables.ids, r[ok], "expand_emit: block_ids")
        t0 = tok_off[s] + j * bs
        cnt = np.minimum(nn - j * bs, bs)
        ok &= (ids >= 0) & (ids < num_blocks) & (cnt > 0) & (t0 >= 0) & (t0 + cnt <= total_tokens)
        part = np.zeros((b.size, 4), np.int64)
        part[ok] = np.stack([ids[ok], t0[ok], cnt[ok], s[ok]], axis=1)
        if (part > INT32_MAX).any() or (part < 0).any():
            raise ModelError("expand_emit: a descriptor field leaves int32")
        desc[b[0]:b[-1] + 1] = part
        if not ok.all():
            flag = 1
        mem.store(desc_addr + 16 * b, desc[b[0]:b[-1] + 1].view(np.uint8).reshape(-1, 16),
                  "expand_emit: descriptors")
        if bucket_addr is not None:
            bk = bucket_of(part[:, 0], num_blocks if num_blocks > 0 else 1, nb)
            mem.load_i32(bucket_addr, np.unique(bk), "expand_emit: bucket count")
    return Expanded(desc, tok_off, blk_off, flag)


def bucket_of(block: np.ndarray, num_blocks: int, nb: int) -> np.ndarray:
    b = np.maximum(np.asarray(block, np.int64), 0) * nb // num_blocks
    return np.minimum(b, nb - 1)


def sort_buckets(n_desc: int) -> int:
    return (max(n_desc, 1) + DESCS_PER_BUCKET - 1) // DESCS_PER_BUCKET


def sort_new(mem: Mem, desc: np.ndarray, num_blocks: int, bucket_addr: int, sorted_addr: int,
             rng: np.random.Generator) -> np.ndarray:
    """sort_scan + sort_scatter: counts per bucket, exclusive scan, then every descriptor placed by an
    atomic increment of its bucket's cursor (arrival order drawn at random: any order must do)."""
    n = len(desc)
    if n == 0:
        return desc
    nb = sort_buckets(n)
    bk = bucket_of(desc[:, 0], max(num_blocks, 1), nb)
    cnt = np.bincount(bk, minlength=nb)
    cursor = np.concatenate([[0], np.cumsum(cnt)[:-1]])
    mem.store_i32(bucket_addr, np.arange(nb), np.zeros(nb), "sort_scan: counters")   # rewritten in place
    # the lanes' atomic increments arrive in a random order; lane i takes its bucket's cursor and advances it,
    # so within a bucket positions follow the arrival order: a stable sort of the arrival order by bucket
    arrival = rng.permutation(n)
    order = arrival[np.argsort(bk[arrival], kind="stable")]
    del arrival
    pos = np.empty(n, np.int64)
    pos[order] = np.arange(n, dtype=np.int64)
    del order
    if not ((pos >= 0) & (pos < n)).all() or (np.bincount(pos, minlength=n) != 1).any():
        raise ModelError("sort_scatter positions are not a permutation")
    if ((pos < cursor[bk]) | (pos >= cursor[bk] + cnt[bk])).any():
        raise ModelError("sort_scatter position outside its bucket's range")
    out = np.zeros_like(desc)
    out[pos] = desc
    d = np.ascontiguousarray(desc, dtype=np.int32)
    mem.store(sorted_addr + 16 * pos, d.view(np.uint8).reshape(-1, 16), "sort_scatter: sorted descriptors")
    return out


# ---------------------------------------------------------------------------
# launch decisions (the host launch code's choices)
# ---------------------------------------------------------------------------

@dataclass
class Slice:
    """One staging slice of a call (HostSlice): addresses already offset to the slice's first head."""
    paged_k: int
    paged_v: int
    stage: int
    row_bytes: int
    layer: int
    head_local: int
    head_count: int
    layer_k: int
    layer_v: int


@dataclass
class Launch:
    kernel: str
    grid: Tuple[int, int]
    threads: int
    unroll: int
    xcd: bool
    args: dict = field(default_factory=dict)


def copy_launches(slices: Sequence[Slice], n_desc: int, bs: int, block_stride: int, row_stride: int,
                  total_tokens: int, pack: bool, wg_bytes: int = 0) -> List[Launch]:
    """launch_copy: vector width, units per workgroup, one launch per 8 slices."""
    if not slices or n_desc == 0:
        return []
    bits = block_stride | row_stride | 16
    max_row = 0
    partial = False
    for s in slices:
        bits |= s.paged_k | s.paged_v | s.stage | s.row_bytes | (total_tokens * s.row_bytes)
        max_row = max(max_row, s.row_bytes)
        partial |= s.row_bytes < row_stride
    vec = lowest_bit(bits)
    per_unit = bs * max_row
    small = per_unit <= SMALL_UNIT_BYTES
    target = wg_bytes or (SMALL_WG_BYTES if small else LARGE_WG_BYTES)
    C = max(1, min(MAX_UNITS_PER_WG, target // per_unit))
    while C > 1 and C * bs * (max_row // vec) >= MAX_WG_VECTORS:
        C >>= 1
    if bs * (max_row // vec) >= MAX_WG_VECTORS:
        raise ModelError("unsupported: a block exceeds the workgroup index space")
    gx = (2 * n_desc + C - 1) // C
    tiny = not pack and C * per_unit <= UNPACK_TINY_WG_BYTES
    shape = ((PACK_PARTIAL if partial else PACK_SMALL) if pack else (UNPACK_TINY if tiny else UNPACK_SMALL)) \
        if small else LARGE
    check_grid(gx, MAX_ITEMS, shape[0], "copy")
    out = []
    for f in range(0, len(slices), MAX_ITEMS):
        group = list(slices[f:f + MAX_ITEMS])
        out.append(Launch("copy_slices", (gx, len(group)), *shape,
                          args=dict(items=group, vec=vec, C=C, bs=bs, block_stride=block_stride,
                                    row_stride=row_stride, total_tokens=total_tokens, n_desc=n_desc, pack=pack)))
    return out


def merged_rows_groups(slices: Sequence[Slice], heads_per_rank: int, min_seg: int,
                       max_seg: int) -> Optional[List[List[Slice]]]:
    """merged_rows_apply: per layer, 2..4 equal slices tiling the rank's heads, the same split in every layer."""
    layers = []
    for s in slices:
        if s.layer not in layers:
            layers.append(s.layer)
    groups: List[List[Slice]] = []
    for l in layers:
        g = sorted((s for s in slices if s.layer == l), key=lambda s: s.head_local)
        if not 2 <= len(g) <= MAX_MERGE_SEGS:
            return None
        nxt = 0
        for s in g:
            if s.head_local != nxt or not min_seg <= s.row_bytes <= max_seg or s.head_count != g[0].head_count:
                return None
            nxt += s.head_count
        if nxt != heads_per_rank:
            return None
        if groups and [(s.head_local, s.head_count) for s in g] != [(s.head_local, s.head_count) for s in groups[0]]:
            return None
        groups.append(g)
    return groups or None


def rows_launches(groups: List[List[Slice]], n_desc: int, bs: int, block_stride: int, row_stride: int,
                  total_tokens: int, pack: bool, wg_bytes: int = 0) -> List[Launch]:
    if not groups or n_desc == 0:
        return []
    nseg = len(groups[0])
    seg_bytes = groups[0][0].row_bytes
    if nseg * seg_bytes != row_stride:
        raise ModelError("whole-row shares do not tile the row")
    bits = block_stride | row_stride | seg_bytes | 16
    for g in groups:
        for s in g:
            bits |= s.layer_k | s.layer_v | s.stage | s.row_bytes | (total_tokens * s.row_bytes)
    vec = lowest_bit(bits)
    per_unit = bs * row_stride
    small = per_unit <= SMALL_UNIT_BYTES
    target = wg_bytes or (SMALL_WG_BYTES if small else LARGE_WG_BYTES)
    C = max(1, min(MAX_UNITS_PER_WG, target // per_unit))
    while C > 1 and C * bs * (row_stride // vec) >= MAX_WG_VECTORS:
        C >>= 1
    if bs * (row_stride // vec) >= MAX_WG_VECTORS:
        raise ModelError("unsupported: a block of one row exceeds the workgroup index space")
    gx = (2 * n_desc + C - 1) // C
    check_grid(gx, MAX_MERGE_GROUPS, (ROWS_SMALL if small else ROWS_LARGE)[0], "whole rows")
    out = []
    for f in range(0, len(groups), MAX_MERGE_GROUPS):
        gg = groups[f:f + MAX_MERGE_GROUPS]
        out.append(Launch("copy_rows", (gx, len(gg)), *(ROWS_SMALL if small else ROWS_LARGE),
                          args=dict(groups=gg, vec=vec, C=C, bs=bs, block_stride=block_stride, row_stride=row_stride,
                                    seg_bytes=seg_bytes, nseg=nseg, total_tokens=total_tokens, n_desc=n_desc,
                                    pack=pack)))
    return out


def tile_launches(slices: Sequence[Slice], n_desc: int, bs: int, block_stride: int, hb: int, eb: int, layout: int,
                  total_tokens: int, pack: bool) -> List[Launch]:
    if not slices or n_desc == 0:
        return []
    bits = block_stride | hb
    max_hc = 1
    for s in slices:
        bits |= s.paged_k | s.paged_v | s.stage
        max_hc = max(max_hc, s.row_bytes // hb)
    if bits & 15:
        raise ModelError("unsupported: head tiles need 16-byte alignment")
    tile_bytes, lrow = bs * hb, hb + 16
    tile_lds = bs * lrow
    if tile_lds > TILE_LDS_BYTES:
        raise ModelError("unsupported: a tile does not fit in LDS")
    tpw = max(1, min(TILE_WG_BYTES // tile_bytes, TILE_LDS_BYTES // tile_lds, MAX_UNITS_PER_WG))
    gx = (n_desc * 2 * max_hc + tpw - 1) // tpw
    check_grid(gx, MAX_ITEMS, TILE_THREADS, "head tiles")
    out = []
    for f in range(0, len(slices), MAX_ITEMS):
        group = list(slices[f:f + MAX_ITEMS])
        out.append(Launch("copy_tiles", (gx, len(group)), TILE_THREADS, 1, False,
                          args=dict(items=group, tpw=tpw, bs=bs, hb=hb, eb=eb, layout=layout, lrow=lrow,
                                    block_stride=block_stride, total_tokens=total_tokens, n_desc=n_desc, pack=pack,
                                    lds_bytes=tpw * tile_lds)))
    return out


@dataclass
class LocalItem:
    src_k: int
    src_v: int
    dst_k: int
    dst_v: int
    row_bytes: int


def local_launches(items: Sequence[LocalItem], n_new: int, bo: int, bn: int, orow: int, nrow: int,
                   wg_bytes: int = 0) -> List[Launch]:
    if not items or n_new == 0:
        return []
    bits = orow | nrow | 16
    max_row = 0
    for it in items:
        bits |= it.src_k | it.src_v | it.dst_k | it.dst_v | it.row_bytes
        max_row = max(max_row, it.row_bytes)
    vec = lowest_bit(bits)
    per_unit = bn * max_row
    small = per_unit <= SMALL_UNIT_BYTES
    target = wg_bytes or (LOCAL_SMALL_WG_BYTES if small else LOCAL_LARGE_WG_BYTES)
    C = max(1, min(MAX_UNITS_PER_WG, target // per_unit))
    C = min(C, max(1, MAX_LOCAL_ROWS // bn))
    if bn > MAX_LOCAL_ROWS:
        raise ModelError("unsupported: new block size above the local-copy row limit")
    while C > 1 and C * bn * (max_row // vec) >= MAX_WG_VECTORS:
        C >>= 1
    if bn * (max_row // vec) >= MAX_WG_VECTORS:
        raise ModelError("unsupported: a block exceeds the workgroup index space")
    gx = (2 * n_new + C - 1) // C
    check_grid(gx, MAX_LOCAL_ITEMS, (LOCAL_SMALL if small else LOCAL_LARGE)[0], "local copy")
    out = []
    for f in range(0, len(items), MAX_LOCAL_ITEMS):
        group = list(items[f:f + MAX_LOCAL_ITEMS])
        out.append(Launch("copy_local", (gx, len(group)), *(LOCAL_SMALL if small else LOCAL_LARGE),
                          args=dict(items=group, vec=vec, C=C, bo=bo, bn=bn, orow=orow, nrow=nrow, n_new=n_new)))
    return out


def local_tile_launches(items: Sequence[LocalItem], n_new: int, bo: int, bn: int, hb: int, eb: int, lo: int,
                        ln: int, orow: int, nrow: int) -> List[Launch]:
    if not items or n_new == 0:
        return []
    if hb % 16:
        raise ModelError("unsupported: head tiles need head_dim * elem_bytes % 16 == 0")
    if bn > MAX_LOCAL_ROWS:
        raise ModelError("unsupported: new block size above the local-copy row limit")
    lrow = hb + 16
    tile_lds = bn * lrow
    if tile_lds > TILE_LDS_BYTES:
        raise ModelError("unsupported: a head tile does not fit the LDS budget")
    T = max(1, TILE_WG_BYTES // (bn * hb))
    T = min(T, TILE_LDS_BYTES // tile_lds, MAX_LOCAL_ROWS // bn, MAX_UNITS_PER_WG)
    out = []
    for f in range(0, len(items), MAX_LOCAL_ITEMS):
        group = list(items[f:f + MAX_LOCAL_ITEMS])
        max_hc = max(1, max(it.row_bytes // hb for it in group))
        gx = (n_new * 2 * max_hc + T - 1) // T
        check_grid(gx, MAX_LOCAL_ITEMS, TILE_THREADS, "local head tiles")
        out.append(Launch("copy_local_tiles", (gx, len(group)), TILE_THREADS, 1, False,
                          args=dict(items=group, T=T, bo=bo, bn=bn, hb=hb, eb=eb, lo=lo, ln=ln, lrow=lrow,
                                    orow=orow, nrow=nrow, n_new=n_new,
                                    old_head_step=hb if lo == NHD else hb * bo,
                                    new_head_step=hb if ln == NHD else hb * bn, lds_bytes=T * tile_lds)))
    return out


# ---------------------------------------------------------------------------
# kernels, vectorized over the launched workgroups (each lane's arithmetic as in the kernel)
# ---------------------------------------------------------------------------

def _flatten(counts) -> Tuple[np.ndarray, np.ndarray]:
    """(owner, local index) of every element when owner i has counts[i] elements."""
    counts = np.asarray(counts, np.int64)
    owner = np.repeat(np.arange(counts.size), counts)
    starts = np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.int64)
    return owner, np.arange(int(counts.sum()), dtype=np.int64) - starts[owner]


def div_checked_v(n: np.ndarray, d: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """div_checked with a divisor per element (each distinct divisor through its own magic number)."""
    n = np.asarray(n, np.int64)
    d = np.broadcast_to(np.asarray(d, np.int64), n.shape)
    q = np.empty_like(n)
    for dv in np.unique(d):
        m = d == dv
        q[m] = div_checked(n[m], int(dv))[0]
    return q, n - q * d


def _desc_load(mem: Mem, desc_addr: int, index: np.ndarray, what: str) -> np.ndarray:
    raw = mem.load(desc_addr + 16 * np.asarray(index, np.int64), 16, what)
    return raw.view(np.int32).reshape(-1, 4).astype(np.int64)


def _check_u32(total: np.ndarray, threads: int, unroll: int, what: str) -> None:
    if (np.asarray(total, np.int64) + threads * unroll >= (1 << 32)).any():
        raise ModelError(f"{what}: 32-bit lane index can wrap")


def _selected(L: Launch, workgroups: Optional[np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """(cx, cy) cells of the selected workgroups (all by default) under the launch's cell order."""
    gx, gy = L.grid
    cxs, cys = grid_cells(gx, gy, L.xcd)
    wgs = np.arange(gx * gy) if workgroups is None else np.asarray(workgroups, np.int64)
    return cxs[wgs], cys[wgs]


class LdsBank:
    """The LDS of many workgroups at once: workgroup w owns bytes [w * size, (w + 1) * size)."""

    def __init__(self, n_wg: int, size: int):
        self.size = size
        self.data = np.full(max(n_wg, 1) * size, 0xA5, np.uint8)   # poison: read only on dead paths

    def _idx(self, w, off, n):
        off = np.asarray(off, np.int64)
        if ((off < 0) | (off + n > self.size)).any():
            raise ModelError(f"LDS access outside the workgroup's {self.size} bytes")
        return (np.asarray(w, np.int64) * self.size + off)[:, None] + np.arange(n)

    def store(self, w, off, vals):
        self.data[self._idx(w, off, vals.shape[1])] = vals

    def load(self, w, off, n):
        return self.data[self._idx(w, off, n)]


def _copy_units(L: Launch, cx, cy, n_desc: int, row_bytes: np.ndarray):
    """Unit ranges of the selected workgroups: (u0, nu) per workgroup, dropping empty ones."""
    C = L.args["C"]
    u0 = cx * C
    nu = np.minimum(C, 2 * n_desc - u0)
    if (nu > MAX_UNITS_PER_WG).any():
        raise ModelError(f"{L.kernel}: more units than its LDS arrays hold")
    keep = nu > 0
    return u0[keep], nu[keep], cy[keep]


def run_copy_slices(mem: Mem, L: Launch, desc_addr: int, workgroups: Optional[np.ndarray] = None) -> None:
    a = L.args
    vec, bs = a["vec"], a["bs"]
    cx, cy = _selected(L, workgroups)
    items = a["items"]
    u0, nu, cy = _copy_units(L, cx, cy, a["n_desc"], None)
    if nu.size == 0:
        return
    rb = np.array([it.row_bytes for it in items], np.int64)[cy]
    pk = np.array([it.paged_k for it in items], np.int64)[cy]
    pv = np.array([it.paged_v for it in items], np.int64)[cy]
    st = np.array([it.stage for it in items], np.int64)[cy]
    vpr = rb // vec
    unit = bs * vpr
    total = nu * unit
    _check_u32(total, L.threads, L.unroll, "copy_slices")
    # prologue: the units' base addresses (the LDS arrays s_paged, s_stage, s_n)
    uw, ul = _flatten(nu)
    g = u0[uw] + ul
    d = _desc_load(mem, desc_addr, g >> 1, "copy_slices: descriptors")
    kv = g & 1
    s_paged = np.where(kv == 1, pv[uw], pk[uw]) + d[:, 0] * a["block_stride"]
    s_stage = st[uw] + kv * a["total_tokens"] * rb[uw] + d[:, 1] * rb[uw]
    first_unit = np.concatenate([[0], np.cumsum(nu)[:-1]])
    # main loop: lane index -> (unit, row, vector)
    ew, idx = _flatten(total)
    u, rem = div_checked_v(idx, unit[ew])
    row, c = div_checked_v(rem, vpr[ew])
    ui = first_unit[ew] + u
    live = row < d[ui, 2]
    paged = (s_paged[ui] + row * a["row_stride"] + c * vec)[live]
    stage = (s_stage[ui] + rem * vec)[live]
    src, dst = (paged, stage) if a["pack"] else (stage, paged)
    mem.store(dst, mem.load(src, vec, "copy_slices: load"), "copy_slices: store")


def run_copy_rows(mem: Mem, L: Launch, desc_addr: int, workgroups: Optional[np.ndarray] = None) -> None:
    a = L.args
    vec, bs, nseg, seg = a["vec"], a["bs"], a["nseg"], a["seg_bytes"]
    cx, cy = _selected(L, workgroups)
    u0, nu, cy = _copy_units(L, cx, cy, a["n_desc"], None)
    if nu.size == 0:
        return
    groups = a["groups"]
    lk = np.array([g[0].layer_k for g in groups], np.int64)[cy]
    lv = np.array([g[0].layer_v for g in groups], np.int64)[cy]
    stg = np.array([[s.stage for s in g] + [0] * (MAX_MERGE_SEGS - len(g)) for g in groups], np.int64)[cy]
    vps = seg // vec
    per_seg = bs * vps
    unit = nseg * per_seg
    total = nu * unit
    _check_u32(total, L.threads, L.unroll, "copy_rows")
    uw, ul = _flatten(nu)
    g = u0[uw] + ul
    d = _desc_load(mem, desc_addr, g >> 1, "copy_rows: descriptors")
    kv = g & 1
    s_paged = np.where(kv == 1, lv[uw], lk[uw]) + d[:, 0] * a["block_stride"]
    first_unit = np.concatenate([[0], np.cumsum(nu)[:-1]])
    ew, idx = _flatten(total)
    u, rem = div_checked(idx, unit)
    sg, r2 = div_checked(rem, per_seg)
    row, cs = div_checked(r2, vps)
    ui = first_unit[ew] + u
    live = row < d[ui, 2]
    base = stg[ew, np.minimum(sg, MAX_MERGE_SEGS - 1)]
    stage = base + kv[ui] * a["total_tokens"] * seg + (d[ui, 1] + row) * seg + cs * vec
    paged = s_paged[ui] + row * a["row_stride"] + (sg * vps + cs) * vec
    src, dst = (paged, stage) if a["pack"] else (stage, paged)
    mem.store(dst[live], mem.load(src[live], vec, "copy_rows: load"), "copy_rows: store")


def _live_prefix(n: np.ndarray, s0: np.ndarray, m: int, has_src: Optional[np.ndarray] = None) -> np.ndarray:
    """Live elements of a dim-major vector holding rows s0 .. s0+m-1: min(m, n - s0), cut at the first row
    without a source when has_src ([vectors, m]) is given."""
    live = np.clip(n - s0, None, m)
    if has_src is not None:
        ok = (np.arange(m)[None, :] < live[:, None]) & has_src
        live = np.where(live > 0, np.cumprod(ok, axis=1).sum(axis=1), live)
    return live


def _check_flag_reads(T: int, bn: int, lrow: int, tile: np.ndarray, s0: np.ndarray, m: int, what: str):
    """copy_local_tiles reads a ROCm V vector's m one-byte source flags as one 4-byte (m = 4) or one or two
    8-byte LDS words at byte tile * bn + s0 of the flag array, which follows the tiles (T * bn * lrow
    bytes), the 8-byte source bases and the 4-byte slots (T * bn rows each) in the dynamic LDS: the
    read must be aligned to its word and stay within the tile's own rows."""
    rows_cap = T * bn
    base = rows_cap * lrow
    word = 4 if m == 4 else 8
    off = base + rows_cap * 12 + tile * bn + s0
    if base % 8 or (off % word).any() or (s0 + m > bn).any() or (s0 < 0).any():
        raise ModelError(f"{what}: a vector's source flags are not aligned words within its tile's rows")


def _store_prefixes(mem: Mem, dst: np.ndarray, vals: np.ndarray, live: np.ndarray, eb: int, m: int, what: str):
    for k in range(1, m + 1):
        sel = live == k
        if sel.any():
            mem.store(dst[sel], vals[sel][:, :k * eb], what)


def run_copy_tiles(mem: Mem, L: Launch, desc_addr: int, workgroups: Optional[np.ndarray] = None) -> None:
    a = L.args
    gx, gy = L.grid
    tpw, bs, hb, eb, layout, lrow = a["tpw"], a["bs"], a["hb"], a["eb"], a["layout"], a["lrow"]
    tile_bytes, vph, m = bs * hb, hb // 16, 16 // eb
    vpt = tile_bytes // 16
    tile_lds = bs * lrow
    wgs = np.arange(gx * gy) if workgroups is None else np.asarray(workgroups, np.int64)
    bx, by = wgs % gx, wgs // gx
    hc = np.array([it.row_bytes // hb for it in a["items"]], np.int64)[by]
    ntiles = a["n_desc"] * 2 * hc
    g0 = bx * tpw
    keep = g0 < ntiles
    bx, by, hc, ntiles, g0 = bx[keep], by[keep], hc[keep], ntiles[keep], g0[keep]
    if bx.size == 0:
        return
    nt = np.minimum(tpw, ntiles - g0)
    _check_u32(nt * vpt, TILE_THREADS, 1, "copy_tiles")
    items = a["items"]
    rb = np.array([it.row_bytes for it in items], np.int64)[by]
    pk = np.array([it.paged_k for it in items], np.int64)[by]
    pv = np.array([it.paged_v for it in items], np.int64)[by]
    st = np.array([it.stage for it in items], np.int64)[by]
    # prologue per tile
    tw, ti = _flatten(nt)
    g = g0[tw] + ti
    dd = g // (2 * hc[tw])
    r = g - dd * 2 * hc[tw]
    kv, j = r // hc[tw], r % hc[tw]
    d = _desc_load(mem, desc_addr, dd, "copy_tiles: descriptors")
    s_paged = np.where(kv == 1, pv[tw], pk[tw]) + d[:, 0] * a["block_stride"] + j * tile_bytes
    s_stage = st[tw] + kv * a["total_tokens"] * rb[tw] + d[:, 1] * rb[tw] + j * hb
    n = d[:, 2]
    lds = LdsBank(bx.size, a["lds_bytes"])
    # every (tile, vector)
    xt, v = _flatten(np.full(tw.size, vpt))
    w_, tl = tw[xt], ti[xt] * tile_lds
    nn, kk = n[xt], kv[xt]
    srow, cb = div_checked(v, vph)
    rowv = srow < nn
    if a["pack"]:
        src = s_paged[xt] + v * 16
        if layout == HND:
            lds.store(w_[rowv], tl[rowv] + srow[rowv] * lrow + cb[rowv] * 16,
                      mem.load(src[rowv], 16, "copy_tiles: pool load"))
        else:
            c, sr = div_checked(v, bs)
            kmask = (kk == 0) & (sr < nn)
            lds.store(w_[kmask], tl[kmask] + sr[kmask] * lrow + c[kmask] * 16,
                      mem.load(src[kmask], 16, "copy_tiles: pool load"))
            dim, s0 = div_checked(v * m, bs)
            vmask = (kk == 1) & (s0 < nn)
            vals = mem.load(src[vmask], 16, "copy_tiles: pool load").reshape(-1, m, eb)
            offs = (tl[vmask] + dim[vmask] * eb)[:, None] + (s0[vmask][:, None] + np.arange(m)) * lrow
            lds.store(np.repeat(w_[vmask], m), offs.reshape(-1), vals.reshape(-1, eb))
        mem.store(s_stage[xt][rowv] + srow[rowv] * rb[tw][xt][rowv] + cb[rowv] * 16,
                  lds.load(w_[rowv], tl[rowv] + srow[rowv] * lrow + cb[rowv] * 16, 16), "copy_tiles: staging store")
        return
    lds.store(w_[rowv], tl[rowv] + srow[rowv] * lrow + cb[rowv] * 16,
              mem.load(s_stage[xt][rowv] + srow[rowv] * rb[tw][xt][rowv] + cb[rowv] * 16, 16,
                       "copy_tiles: staging load"))
    dst = s_paged[xt] + v * 16
    if layout == HND:
        mem.store(dst[rowv], lds.load(w_[rowv], tl[rowv] + srow[rowv] * lrow + cb[rowv] * 16, 16),
                  "copy_tiles: pool store")
        return
    c, sr = div_checked(v, bs)
    kmask = (kk == 0) & (sr < nn)
    mem.store(dst[kmask], lds.load(w_[kmask], tl[kmask] + sr[kmask] * lrow + c[kmask] * 16, 16),
              "copy_tiles: pool store")
    dim, s0 = div_checked(v * m, bs)
    live = _live_prefix(nn, s0, m)
    vmask = (kk == 1) & (live > 0)
    offs = (tl[vmask] + dim[vmask] * eb)[:, None] + (s0[vmask][:, None] + np.arange(m)) * lrow
    vals = lds.load(np.repeat(w_[vmask], m), offs.reshape(-1), eb).reshape(-1, 16)
    _store_prefixes(mem, dst[vmask], vals, live[vmask], eb, m, "copy_tiles: pool store")


def _resolve_rows(mem: Mem, d: np.ndarray, rows: np.ndarray, tok_off_addr: int, blk_off_addr: int,
                  old_desc_addr: int, n_old: int, bo: int):
    """The local copies' prologue for (descriptor, row) pairs: (ok, old descriptor, slot, flag)."""
    live = rows < d[:, 2]
    seq = d[:, 3]
    t = np.zeros(len(d), np.int64)
    ob = np.zeros(len(d), np.int64)
    slot = np.zeros(len(d), np.int64)
    ok = live.copy()
    if live.any():
        to = mem.load_i32(tok_off_addr, seq[live], "copy_local: token offsets")
        bo_ = mem.load_i32(blk_off_addr, seq[live], "copy_local: old block offsets")
        t[live] = d[live, 1] - to + rows[live]
        q = cdiv_trunc(t[live], bo)
        ob[live] = bo_ + q
        slot[live] = t[live] - q * bo
    ok &= (t >= 0) & (ob >= 0) & (ob < n_old)
    od = np.zeros((len(d), 4), np.int64)
    if ok.any():
        od[ok] = _desc_load(mem, old_desc_addr, ob[ok], "copy_local: old descriptors")
    ok &= (od[:, 3] == seq) & (slot < od[:, 2])
    flag = bool((live & ~ok).any())
    return ok, od, slot, flag


def run_copy_local(mem: Mem, L: Launch, ws: dict, workgroups: Optional[np.ndarray] = None) -> int:
    a = L.args
    vec, bo, bn = a["vec"], a["bo"], a["bn"]
    cx, cy = _selected(L, workgroups)
    u0, nu, cy = _copy_units(L, cx, cy, a["n_new"], None)
    if nu.size == 0:
        return 0
    if (nu * bn > MAX_LOCAL_ROWS).any():
        raise ModelError("copy_local: more rows than its LDS array holds")
    items = a["items"]
    rb = np.array([it.row_bytes for it in items], np.int64)[cy]
    sk = np.array([it.src_k for it in items], np.int64)[cy]
    sv = np.array([it.src_v for it in items], np.int64)[cy]
    dk = np.array([it.dst_k for it in items], np.int64)[cy]
    dv = np.array([it.dst_v for it in items], np.int64)[cy]
    uw, ul = _flatten(nu)
    g = u0[uw] + ul
    d = _desc_load(mem, ws["sorted_new"], g >> 1, "copy_local: new descriptors")
    kv = g & 1
    s_dst = np.where(kv == 1, dv[uw], dk[uw]) + d[:, 0] * (a["nrow"] * bn)
    # row prologue: unit-major (unit, row) pairs, bn rows per unit
    ru, rr = _flatten(np.full(uw.size, bn))
    ok, od, slot, flag = _resolve_rows(mem, d[ru], rr, ws["scan_old"], ws["scan_old"] + 4 * (ws["S"] + 1),
                                       ws["desc_old"], ws["n_old"], bo)
    s_src = np.where(ok, np.where(kv[ru] == 1, sv[uw][ru], sk[uw][ru]) + od[:, 0] * (a["orow"] * bo) +
                     slot * a["orow"], 0)
    vpr = rb // vec
    unit = bn * vpr
    total = nu * unit
    _check_u32(total, L.threads, L.unroll, "copy_local")
    first_unit = np.concatenate([[0], np.cumsum(nu)[:-1]])
    ew, idx = _flatten(total)
    u, rem = div_checked_v(idx, unit[ew])
    row, c = div_checked_v(rem, vpr[ew])
    ui = first_unit[ew] + u
    src_row = s_src[ui * bn + row]
    live = (row < d[ui, 2]) & (src_row != 0)
    dst = (s_dst[ui] + row * a["nrow"] + c * vec)[live]
    mem.store(dst, mem.load((src_row + c * vec)[live], vec, "copy_local: load"), "copy_local: store")
    return int(flag)


def run_copy_local_tiles(mem: Mem, L: Launch, ws: dict, workgroups: Optional[np.ndarray] = None) -> int:
    a = L.args
    gx, gy = L.grid
    T, bo, bn, hb, eb, lo, ln, lrow = a["T"], a["bo"], a["bn"], a["hb"], a["eb"], a["lo"], a["ln"], a["lrow"]
    vph, m = hb // 16, 16 // eb
    per_tile = bn * vph
    tile_lds = bn * lrow
    wgs = np.arange(gx * gy) if workgroups is None else np.asarray(workgroups, np.int64)
    bx, by = wgs % gx, wgs // gx
    items = a["items"]
    hc = np.array([it.row_bytes // hb for it in items], np.int64)[by]
    ntiles = a["n_new"] * 2 * hc
    g0 = bx * T
    keep = g0 < ntiles
    bx, by, hc, ntiles, g0 = bx[keep], by[keep], hc[keep], ntiles[keep], g0[keep]
    if bx.size == 0:
        return 0
    nt = np.minimum(T, ntiles - g0)
    if (nt * bn > MAX_LOCAL_ROWS).any():
        raise ModelError("copy_local_tiles: more rows than its LDS arrays hold")
    _check_u32(nt * per_tile, TILE_THREADS, 1, "copy_local_tiles")
    sk = np.array([it.src_k for it in items], np.int64)[by]
    sv = np.array([it.src_v for it in items], np.int64)[by]
    dk = np.array([it.dst_k for it in items], np.int64)[by]
    dv = np.array([it.dst_v for it in items], np.int64)[by]
    tw, ti = _flatten(nt)
    g = g0[tw] + ti
    dd = g // (2 * hc[tw])
    r = g - dd * 2 * hc[tw]
    kv, j = r // hc[tw], r % hc[tw]
    d = _desc_load(mem, ws["sorted_new"], dd, "copy_local_tiles: new descriptors")
    s_dst = np.where(kv == 1, dv[tw], dk[tw]) + d[:, 0] * (a["nrow"] * bn) + j * a["new_head_step"]
    n = d[:, 2]
    rt, rr = _flatten(np.full(tw.size, bn))            # (tile, row)
    ok, od, slot, flag = _resolve_rows(mem, d[rt], rr, ws["scan_old"], ws["scan_old"] + 4 * (ws["S"] + 1),
                                       ws["desc_old"], ws["n_old"], bo)
    s_src = np.where(ok, np.where(kv[rt] == 1, sv[tw][rt], sk[tw][rt]) + od[:, 0] * (a["orow"] * bo) +
                     j[rt] * a["old_head_step"], 0).reshape(-1, bn)
    s_slot = np.where(ok, slot, 0).reshape(-1, bn)
    has_src = s_src != 0
    xt, v = _flatten(np.full(tw.size, per_tile))       # (tile, vector)
    nn, kk = n[xt], kv[xt]
    if lo == ln and bo == bn:                            # same layout and block size: vector for vector
        src0 = s_src[xt, 0]
        if ln == HND:
            rows = v // vph
        else:
            rows = v - (v // bn) * bn
        plain = (ln == HND) | (kk == 0)
        okv = plain & (src0 != 0) & (rows < nn) & has_src[xt, np.minimum(rows, bn - 1)]
        mem.store(s_dst[xt][okv] + v[okv] * 16, mem.load(src0[okv] + v[okv] * 16, 16, "copy_local_tiles: load"),
                  "copy_local_tiles: store")
        if ln == ROCM:
            dim, s0 = div_checked(v * m, bn)
            vv = (kk == 1) & (src0 != 0)
            _check_flag_reads(T, bn, lrow, ti[xt][vv], s0[vv], m, "copy_local_tiles")
            rowsk = np.minimum(s0[:, None] + np.arange(m), bn - 1)
            live = _live_prefix(nn, s0, m, has_src[xt[:, None], rowsk])
            vm = (kk == 1) & (src0 != 0) & (live > 0)
            vals = mem.load(src0[vm] + v[vm] * 16, 16, "copy_local_tiles: load")
            _store_prefixes(mem, s_dst[xt][vm] + v[vm] * 16, vals, live[vm], eb, m, "copy_local_tiles: store")
        return int(flag)
    if lo == ln:                                         # same layout, block sizes differ: vector from vector
        if ln == HND:
            rows, c = div_checked(v, vph)
            off, sb = c * 16, hb
        else:
            c, rows = div_checked(v, bn)
            off, sb = c * bo * 16, 16
        plain = (ln == HND) | (kk == 0)
        okv = plain & (rows < nn) & has_src[xt, rows]
        src = s_src[xt, rows] + off + s_slot[xt, rows] * sb
        mem.store(s_dst[xt][okv] + v[okv] * 16, mem.load(src[okv], 16, "copy_local_tiles: load"),
                  "copy_local_tiles: store")
        if ln == ROCM:
            dim, s0 = div_checked(v * m, bn)
            vv = kk == 1
            _check_flag_reads(T, bn, lrow, ti[xt][vv], s0[vv], m, "copy_local_tiles")
            rowsk = np.minimum(s0[:, None] + np.arange(m), bn - 1)
            live = _live_prefix(nn, s0, m, has_src[xt[:, None], rowsk])
            slot0 = s_slot[xt, s0]
            vm = vv & (live > 0) & (slot0 % m == 0)
            vals = mem.load(s_src[xt, s0][vm] + dim[vm] * bo * eb + slot0[vm] * eb, 16, "copy_local_tiles: load")
            _store_prefixes(mem, s_dst[xt][vm] + v[vm] * 16, vals, live[vm], eb, m, "copy_local_tiles: store")
        return int(flag)
    lds = LdsBank(bx.size, a["lds_bytes"])
    w_, tl = tw[xt], ti[xt] * tile_lds
    rows, c = div_checked(v, vph)
    base = s_src[xt, rows]
    okr = (rows < nn) & (base != 0)
    sl = s_slot[xt, rows]
    if lo == NHD:
        val = mem.load(base[okr] + sl[okr] * a["orow"] + c[okr] * 16, 16, "copy_local_tiles: load")
    elif lo == HND:
        val = mem.load(base[okr] + sl[okr] * hb + c[okr] * 16, 16, "copy_local_tiles: load")
    else:
        # K tiles as the other layouts; V tiles ([dim][slot]) by vectors of m rows of one dim (below)
        okk = okr & (kk == 0)
        val = mem.load(base[okk] + c[okk] * bo * 16 + sl[okk] * 16, 16, "copy_local_tiles: load")
    if lo != ROCM:
        lds.store(w_[okr], tl[okr] + rows[okr] * lrow + c[okr] * 16, val)
    else:
        lds.store(w_[okk], tl[okk] + rows[okk] * lrow + c[okk] * 16, val)
    if lo == ROCM:
        vv = kk == 1
        dim, s0 = div_checked(v * m, bn)
        nl = np.minimum(m, nn - s0)
        _check_flag_reads(T, bn, lrow, ti[xt][vv & (nl > 0)], s0[vv & (nl > 0)], m, "copy_local_tiles")
        rowsk = np.minimum(s0[:, None] + np.arange(m), bn - 1)
        run = _live_prefix(nn, s0, m, has_src[xt[:, None], rowsk])
        slot0 = s_slot[xt, s0]
        run = np.where(slot0 % m == 0, run, 0)
        vm = vv & (nl > 0) & (run > 0)
        vals = mem.load(s_src[xt, s0][vm] + dim[vm] * bo * eb + slot0[vm] * eb, 16, "copy_local_tiles: load")
        offs = (tl[vm] + dim[vm] * eb)[:, None] + (s0[vm][:, None] + np.arange(m)) * lrow
        lds.store(np.repeat(w_[vm], m), offs.reshape(-1), vals.reshape(-1, eb))
        for k in range(m):                               # live rows outside the run, element by element
            r_ = np.minimum(s0 + k, bn - 1)
            em = vv & (k >= np.maximum(run, 0)) & (k < nl) & has_src[xt, r_]
            if em.any():
                e = mem.load(s_src[xt, r_][em] + dim[em] * bo * eb + s_slot[xt, r_][em] * eb, eb,
                             "copy_local_tiles: load")
                lds.store(w_[em], tl[em] + (s0[em] + k) * lrow + dim[em] * eb, e)
    if ln == NHD:
        mem.store(s_dst[xt][okr] + rows[okr] * a["nrow"] + c[okr] * 16,
                  lds.load(w_[okr], tl[okr] + rows[okr] * lrow + c[okr] * 16, 16), "copy_local_tiles: store")
        return int(flag)
    dst = s_dst[xt] + v * 16
    if ln == HND:
        mem.store(dst[okr], lds.load(w_[okr], tl[okr] + rows[okr] * lrow + c[okr] * 16, 16),
                  "copy_local_tiles: store")
        return int(flag)
    cK, rK = div_checked(v, bn)
    kmask = (kk == 0) & (rK < nn) & has_src[xt, rK]
    mem.store(dst[kmask], lds.load(w_[kmask], tl[kmask] + rK[kmask] * lrow + cK[kmask] * 16, 16),
              "copy_local_tiles: store")
    dim, s0 = div_checked(v * m, bn)
    _check_flag_reads(T, bn, lrow, ti[xt][kk == 1], s0[kk == 1], m, "copy_local_tiles")
    rowsk = np.minimum(s0[:, None] + np.arange(m), bn - 1)
    live = _live_prefix(nn, s0, m, has_src[xt[:, None], rowsk])
    vm = (kk == 1) & (live > 0)
    offs = (tl[vm] + dim[vm] * eb)[:, None] + (s0[vm][:, None] + np.arange(m)) * lrow
    vals = lds.load(np.repeat(w_[vm], m), offs.reshape(-1), eb).reshape(-1, 16)
    _store_prefixes(mem, dst[vm], vals, live[vm], eb, m, "copy_local_tiles: store")
    return int(flag)


def run_launch(mem: Mem, L: Launch, ws: dict, desc_addr: Optional[int] = None,
               workgroups: Optional[np.ndarray] = None) -> int:
    if L.kernel == "copy_slices":
        run_copy_slices(mem, L, desc_addr, workgroups)
    elif L.kernel == "copy_rows":
        run_copy_rows(mem, L, desc_addr, workgroups)
    elif L.kernel == "copy_tiles":
        run_copy_tiles(mem, L, desc_addr, workgroups)
    elif L.kernel == "copy_local":
        return run_copy_local(mem, L, ws, workgroups)
    elif L.kernel == "copy_local_tiles":
        return run_copy_local_tiles(mem, L, ws, workgroups)
    else:
        raise ValueError(L.kernel)
    return 0


# ---------------------------------------------------------------------------
# a migration through the model
# ---------------------------------------------------------------------------

def _align256(x: int) -> int:
    return (x + 255) // 256 * 256


def workspace_layout(S: int, old_live: int, new_live: int) -> dict:
    """Byte offsets of the workspace areas (header, scans, descriptors, sort counters, sorted descriptors)."""
    scan = _align256(2 * (S + 1) * 4)
    out = {"stamp_old": 8, "stamp_new": 16, "scan_old": 256}
    out["scan_new"] = out["scan_old"] + scan
    out["desc_old"] = out["scan_new"] + scan
    out["desc_new"] = out["desc_old"] + _align256(max(old_live, 1) * 16)
    out["bucket_new"] = out["desc_new"] + _align256(max(new_live, 1) * 16)
    out["sorted_new"] = out["bucket_new"] + _align256(max(new_live, 1) * 4)
    out["total"] = out["sorted_new"] + _align256(max(new_live, 1) * 16)
    return out


@dataclass
class _Topo:
    tp: int
    pp: int
    starts: List[int]
    H: int

    @classmethod
    def of(cls, t, L: int, H: int) -> "_Topo":
        tp, pp = int(t[0]), int(t[1])
        starts = list(t[2]) if len(t) > 2 and t[2] is not None else [p * L // pp for p in range(pp + 1)]
        return cls(tp, pp, starts, H)

    def first_layer(self, r: int) -> int:
        return self.starts[r // self.tp]

    def layers(self, r: int) -> range:
        return range(self.starts[r // self.tp], self.starts[r // self.tp + 1])

    def heads_per_rank(self) -> int:
        return self.H // self.tp if self.tp <= self.H else 1

    def first_head(self, r: int) -> int:
        return (r % self.tp) * self.H // self.tp


class Migration:
    """One workload's migration through the model.

    Pools (in any layout), staging, device tables and the workspace live in a
    Mem.  With data=True the pools hold the generated bytes and the result can
    be compared with the oracle; with data=False every pool and staging buffer
    is virtual and only access bounds are checked (full-size launch shapes).
    dev_old / dev_new replace the device copies of the tables (lens, offsets,
    ids) to model tables that disagree with the host ones.
    """

    def __init__(self, w, inp, old_layout: int = NHD, new_layout: int = NHD, data: bool = True,
                 wg_bytes: int = 0, dev_old=None, dev_new=None, seed: int = 0):
        import oracle
        import paper_2606_18741_amd as rk
        import hostpools

        self.w, self.inp = w, inp
        L, H, D, e = w.num_layers, w.num_kv_heads, w.head_dim, w.elem_bytes
        self.L, self.H, self.hrow, self.eb = L, H, D * e, e
        self.lo, self.ln = old_layout, new_layout
        self.wg_bytes = wg_bytes
        self.rng = np.random.default_rng(seed)
        self.plan = rk.Plan(w.old_topo, w.new_topo, (L, H, D, e, w.old_block_size, w.new_block_size),
                            rk.HostTables.of(inp.old_tables))
        info = self.plan.info
        self.T, self.n_old, self.n_new = info.total_tokens, info.old_live_blocks, info.new_live_blocks
        self.S = len(inp.lens)
        self.old, self.new = _Topo.of(w.old_topo, L, H), _Topo.of(w.new_topo, L, H)
        self.bo, self.bn = w.old_block_size, w.new_block_size
        self.pairs = {(p.src, p.dst): p for p in self.plan.pairs}
        self.offs = {k: self.plan.query(*k)[1] for k in self.pairs}
        self.mem = Mem()
        mem = self.mem

        def tables(t, dev, name):
            lens, offs, ids = dev if dev is not None else (t.seq_lens, t.offsets, t.ids)
            return Tables(mem.add(name + "_lens", np.asarray(lens, np.int32)),
                          mem.add(name + "_offs", np.asarray(offs, np.int32)),
                          mem.add(name + "_ids", np.asarray(ids, np.int32)))
        self.dt_old = tables(inp.old_tables, dev_old, "old_tables")
        self.dt_new = tables(inp.new_tables, dev_new, "new_tables")
        self.nnz_old, self.nnz_new = len(inp.old_tables.ids), len(inp.new_tables.ids)
        self.wl = workspace_layout(self.S, self.n_old, self.n_new)
        if self.wl["total"] != self.plan.workspace_bytes:
            raise ModelError("workspace layout differs from the library's")
        self.ws = mem.add("workspace", np.zeros(self.wl["total"], np.uint8))
        self.ws_region = mem.region("workspace")

        # pools: {(side, rank, layer, kv): address}
        self.addr: Dict[tuple, int] = {}
        self.old_host = self.new_host = None
        H_o, H_n = self.old.heads_per_rank(), self.new.heads_per_rank()
        if data:
            self.old_host = hostpools.source_pools(w, inp.old_tables)
            self.new_host = hostpools.sentinel_pools(w, inp.new_tables)
            self.phys = {}
            for side, pools, lay in (("o", self.old_host, old_layout), ("n", self.new_host, new_layout)):
                for r, per in pools.items():
                    for l, a in per.items():
                        kvs = oracle.encode_pool(a, lay)
                        for kv in range(2):
                            self.phys[(side, r, l, kv)] = kvs[kv]
                            self.addr[(side, r, l, kv)] = mem.add(f"{side}{r}.l{l}.{'KV'[kv]}", kvs[kv])
        else:
            for side, topo, tb, hl in (("o", self.old, inp.old_tables, H_o), ("n", self.new, inp.new_tables, H_n)):
                nbytes = tb.num_blocks * tb.block_size * hl * self.hrow
                for r in range(topo.tp * topo.pp):
                    for l in topo.layers(r):
                        for kv in range(2):
                            self.addr[(side, r, l, kv)] = mem.add(f"{side}{r}.l{l}.{'KV'[kv]}", size=nbytes)
        self.staging = {}
        for k, p in self.pairs.items():
            nb = p.staging_bytes
            if data:
                self.staging[k] = mem.add(f"stage{k}", np.full(nb, 0xEE, np.uint8))
            else:
                self.staging[k] = mem.add(f"stage{k}", size=nb)
        # Algorithm 1 order: layer, then new tensor rank, then old head range
        self.items = sorted(((p.src, p.dst, l, p.head_begin, p.head_count)
                             for p in self.plan.pairs for l in range(p.layer_begin, p.layer_end)),
                            key=lambda it: (it[2], it[1] % self.new.tp, it[3]))

    # --- expansion -----------------------------------------------------------
    def _expand_old(self) -> Expanded:
        self.ws_region.writes[:] = 0
        return expand(self.mem, self.dt_old, self.S, self.bo, self.nnz_old, self.inp.old_tables.num_blocks, self.T,
                      self.n_old, self.ws + self.wl["scan_old"], self.ws + self.wl["desc_old"])

    def _expand_new(self) -> Expanded:
        self.ws_region.writes[:] = 0
        nb = sort_buckets(self.n_new)
        ex = expand(self.mem, self.dt_new, self.S, self.bn, self.nnz_new, self.inp.new_tables.num_blocks, self.T,
                    self.n_new, self.ws + self.wl["scan_new"], self.ws + self.wl["desc_new"],
                    self.ws + self.wl["bucket_new"], nb)
        self.ws_region.writes[:] = 0
        sort_new(self.mem, ex.desc, self.inp.new_tables.num_blocks, self.ws + self.wl["bucket_new"],
                 self.ws + self.wl["sorted_new"], self.rng)
        return ex

    # --- slices (collect_slices) ---------------------------------------------
    def _slices(self, pack: bool, rank: int, l0: int, l1: int, skip_local: bool) -> List[Slice]:
        topo = self.old if pack else self.new
        lay = self.lo if pack else self.ln
        bs = self.bo if pack else self.bn
        side = "o" if pack else "n"
        out = []
        for (src, dst, l, hb, hc) in self.items:
            if (src if pack else dst) != rank or not l0 <= l < l1:
                continue
            peer = dst if pack else src
            if skip_local and peer == rank:
                continue
            p = self.pairs[(src, dst)]
            ws0 = max(l0, p.layer_begin)
            ptr = self.staging[(src, dst)] + int(self.offs[(src, dst)][l0])
            k, v = self.addr[(side, rank, l, 0)], self.addr[(side, rank, l, 1)]
            hstep = self.hrow if lay == NHD else self.hrow * bs
            hoff = (hb - topo.first_head(rank)) * hstep
            out.append(Slice(k + hoff, v + hoff, ptr + (l - ws0) * p.slice_bytes, hc * self.hrow, l,
                             hb - topo.first_head(rank), hc, k, v))
        return out

    def _run(self, launches: List[Launch], desc_addr: Optional[int], sample: Optional[int]) -> int:
        flag = 0
        ws = {"sorted_new": self.ws + self.wl["sorted_new"], "scan_old": self.ws + self.wl["scan_old"],
              "desc_old": self.ws + self.wl["desc_old"], "S": self.S, "n_old": self.n_old}
        for Lc in launches:
            n = Lc.grid[0] * Lc.grid[1]
            wgs = None
            if sample is not None and n > sample:
                wgs = np.unique(np.concatenate([[0, n - 1], self.rng.choice(n, sample, replace=False)]))
            flag |= run_launch(self.mem, Lc, ws, desc_addr, wgs)
        return flag

    # --- entry points --------------------------------------------------------
    def pack_launches(self, rank: int, l0: int, l1: int, skip_local: bool = False) -> List[Launch]:
        slices = self._slices(True, rank, l0, l1, skip_local)
        hpr = self.old.heads_per_rank()
        row = hpr * self.hrow
        if self.lo == HND and all(s.head_count == 1 for s in slices):
            return copy_launches(slices, self.n_old, self.bo, row * self.bo, self.hrow, self.T, True, self.wg_bytes)
        if self.lo != NHD:
            return tile_launches(slices, self.n_old, self.bo, row * self.bo, self.hrow, self.eb, self.lo, self.T,
                                 True)
        groups = merged_rows_groups(slices, hpr, PACK_ROWS_MIN, PACK_ROWS_MAX)
        if groups:
            return rows_launches(groups, self.n_old, self.bo, row * self.bo, row, self.T, True, self.wg_bytes)
        return copy_launches(slices, self.n_old, self.bo, row * self.bo, row, self.T, True, self.wg_bytes)

    def unpack_launches(self, rank: int, l0: int, l1: int, skip_local: bool = False) -> List[Launch]:
        slices = self._slices(False, rank, l0, l1, skip_local)
        hpr = self.new.heads_per_rank()
        row = hpr * self.hrow
        if self.ln != NHD:
            return tile_launches(slices, self.n_new, self.bn, row * self.bn, self.hrow, self.eb, self.ln, self.T,
                                 False)
        groups = merged_rows_groups(slices, hpr, UNPACK_ROWS_MIN, UNPACK_ROWS_MAX)
        if groups:
            return rows_launches(groups, self.n_new, self.bn, row * self.bn, row, self.T, False, self.wg_bytes)
        return copy_launches(slices, self.n_new, self.bn, row * self.bn, row, self.T, False, self.wg_bytes)

    def local_launches(self, rank: int, l0: int, l1: int) -> List[Launch]:
        items = []
        for (src, dst, l, hb, hc) in self.items:
            if src != rank or dst != rank or not l0 <= l < l1:
                continue
            ostep = self.hrow if self.lo == NHD else self.hrow * self.bo
            nstep = self.hrow if self.ln == NHD else self.hrow * self.bn
            so = (hb - self.old.first_head(rank)) * ostep
            sn = (hb - self.new.first_head(rank)) * nstep
            items.append(LocalItem(self.addr[("o", rank, l, 0)] + so, self.addr[("o", rank, l, 1)] + so,
                                   self.addr[("n", rank, l, 0)] + sn, self.addr[("n", rank, l, 1)] + sn,
                                   hc * self.hrow))
        orow, nrow = self.old.heads_per_rank() * self.hrow, self.new.heads_per_rank() * self.hrow
        if self.lo != NHD or self.ln != NHD:
            return local_tile_launches(items, self.n_new, self.bo, self.bn, self.hrow, self.eb, self.lo, self.ln,
                                       orow, nrow)
        return local_launches(items, self.n_new, self.bo, self.bn, orow, nrow, self.wg_bytes)

    def pack(self, rank: int, l0: int = 0, l1: Optional[int] = None, skip_local: bool = False,
             sample: Optional[int] = None) -> int:
        l1 = self.L if l1 is None else l1
        if l0 == l1 or self.n_old == 0:
            return 0
        flag = self._expand_old().flag
        return flag | self._run(self.pack_launches(rank, l0, l1, skip_local), self.ws + self.wl["desc_old"], sample)

    def unpack(self, rank: int, l0: int = 0, l1: Optional[int] = None, skip_local: bool = False,
               sample: Optional[int] = None) -> int:
        l1 = self.L if l1 is None else l1
        if l0 == l1 or self.n_new == 0:
            return 0
        flag = self._expand_new().flag
        return flag | self._run(self.unpack_launches(rank, l0, l1, skip_local), self.ws + self.wl["sorted_new"],
                                sample)

    def copy_local(self, rank: int, l0: int = 0, l1: Optional[int] = None, sample: Optional[int] = None) -> int:
        l1 = self.L if l1 is None else l1
        if l0 == l1 or self.n_new == 0:
            return 0
        flag = self._expand_old().flag
        ex_new_flag = self._expand_new().flag
        return flag | ex_new_flag | self._run(self.local_launches(rank, l0, l1), None, sample)

    # --- results ---------------------------------------------------------------
    def migrate(self, windows=None, local: bool = False) -> List[int]:
        """Every old rank packs, every new rank unpacks (and with local, every rank in both topologies copies
        its kept slices pool to pool), per layer window.  Returns the flags of the calls."""
        flags = []
        for (l0, l1) in (windows or [(0, self.L)]):
            for r in range(self.old.tp * self.old.pp):
                flags.append(self.pack(r, l0, l1, skip_local=local))
            for q in range(self.new.tp * self.new.pp):
                flags.append(self.unpack(q, l0, l1, skip_local=local))
            if local:
                for r in range(min(self.old.tp * self.old.pp, self.new.tp * self.new.pp)):
                    flags.append(self.copy_local(r, l0, l1))
        return flags

    def new_pools(self) -> Dict[int, Dict[int, np.ndarray]]:
        """The new pools as logical [2, nb, bs, H_loc, D] arrays (decoded from their layout)."""
        import oracle
        out: Dict[int, Dict[int, np.ndarray]] = {}
        for q, per in self.new_host.items():
            out[q] = {}
            for l, a in per.items():
                kvs = [self.phys[("n", q, l, kv)] for kv in range(2)]
                out[q][l] = oracle.decode_pool(kvs, self.ln)
        return out

    def writes(self, name: str) -> np.ndarray:
        return self.mem.region(name).writes
