// GPU side of the KV-cache migration for gfx950: the host launch code and the
// C entry points (pack, unpack, local copy).  The kernels are in kv_expand.hpp
// (block-table expansion, descriptor sort), kv_copy.hpp (pack / unpack copy,
// NHD local copy), kv_tiles.hpp (head tiles through LDS for HND and ROCm pools)
// and kv_rows.hpp (whole-row unpack); all of them build in this one unit.
//
// The copy is pure data movement (no arithmetic on the payload), so it is
// bound by HBM bandwidth.  The layout makes every 16-byte vector of a slice
// have exactly one source and one destination:
//   paged side   [block][slot][local head][head_dim]  (a row run of head_count*head_dim
//                elements at a stride of H_loc*head_dim)
//   staging side [kv][token][head of the overlap][head_dim] (contiguous per block)
// so both directions are coalesced row copies.  A workgroup owns a chunk of
// consecutive block descriptors of one slice; its lanes stride over the
// chunk's flattened (descriptor, kv, slot, vector) space with several 16-byte
// loads in flight before their stores.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_set>
#include <vector>

#include "device_util.hpp"
#include "kv_copy.hpp"
#include "kv_device.hpp"
#include "kv_expand.hpp"
#include "kv_rows.hpp"
#include "kv_tiles.hpp"
#include "plan.hpp"

namespace remp {

// ---------------------------------------------------------------------------
// host launch code
// ---------------------------------------------------------------------------

static thread_local hipEvent_t g_trace_start = nullptr;
static thread_local hipEvent_t g_trace_stop = nullptr;

// Bytes a copy workgroup aims to move: the built-in target of the launch kind, or the plan's
// tuning override (REMP_KV_WG_BYTES when the plan was created).
static int64_t wg_target(const remp_kv_plan_t& p, int64_t builtin) { return p.wg_bytes > 0 ? p.wg_bytes : builtin; }

// Bound on a copy workgroup's flattened (unit, row, vector) index space.
constexpr uint64_t kMaxWgVectors = uint64_t(1) << 31;

// A dispatch counts its work-items in 32 bits per grid dimension, and the XCD cell order numbers the
// workgroups of a launch linearly in 32 bits.
static remp_status check_grid(int64_t gx, int64_t gy, int threads, const char* what) {
    if (gx * threads >= (int64_t(1) << 32) || gx * gy >= (int64_t(1) << 32))
        return fail(REMP_E_UNSUPPORTED, std::string(what) + ": too many workgroups for one launch");
    return REMP_OK;
}

struct HostSlice {
    uint64_t paged_k, paged_v, stage;
    uint32_t row_bytes;
    int32_t layer = 0;        // global layer
    int32_t head_local = 0;   // first head of the slice within the paged rank's heads
    int32_t head_count = 0;
    uint64_t layer_k = 0, layer_v = 0;   // the layer's storage (no head offset)
};


// Descriptor stamps.  The old descriptors are a function of the plan alone
// (its old tables), the new ones of the plan and the new tables given to the
// call, so a stamp is a 64-bit hash of those (never 0, which no expansion
// writes).  Combination step after Boost's hash_combine, finished with the
// SplitMix64 output function (Steele, Lea and Flood, 2014).
static uint64_t mix64(uint64_t h, uint64_t v) { return h ^ (v + 0x9e3779b97f4a7c15ull + (h << 6) + (h >> 2)); }

static uint64_t finish64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    z ^= z >> 31;
    return z ? z : 1;
}

static uint64_t old_stamp(const remp_kv_plan_t& p) { return finish64(mix64(mix64(0, p.serial), 1)); }

static StampCheck no_check(int32_t* flag) {
    StampCheck c;
    c.at[0] = c.at[1] = nullptr;
    c.want[0] = c.want[1] = 0;
    c.flag = flag;
    return c;
}

static uint32_t sort_buckets(int64_t n_desc) {
    return static_cast<uint32_t>((std::max<int64_t>(n_desc, 1) + kDescsPerBucket - 1) / kDescsPerBucket);
}

// Enqueue expansion of `tables` into the workspace areas at scan_off / desc_off;
// `flag` is the status flag (reset first if reset_flag).  With bucket_off >= 0
// the expansion also clears and fills the bucket counters of the descriptor
// sort (new tables only).  A non-NULL stamp_at receives `stamp` in the same
// launch that writes the descriptors.
static remp_status launch_expand(const remp_kv_plan_t& p, const remp_dev_tables& dt, int32_t bs, int64_t nnz,
                                 int64_t num_blocks, int64_t n_desc, char* ws, int32_t* flag, int64_t scan_off,
                                 int64_t desc_off, bool reset_flag, hipStream_t stream, int64_t bucket_off,
                                 uint64_t* stamp_at, uint64_t stamp) {
    if (n_desc >= (int64_t(1) << 30)) return fail(REMP_E_UNSUPPORTED, "more than 2^30 live blocks in one call");
    int32_t* tok_off = reinterpret_cast<int32_t*>(ws + scan_off);
    int32_t* blk_off = tok_off + (p.num_seqs + 1);
    BlockDesc* desc = reinterpret_cast<BlockDesc*>(ws + desc_off);
    int32_t* bucket = bucket_off >= 0 ? reinterpret_cast<int32_t*>(ws + bucket_off) : nullptr;
    const uint32_t nb = bucket ? sort_buckets(n_desc) : 0;
    hipLaunchKernelGGL(expand_scan, dim3(1), dim3(kScanThreads), 0, stream, dt.seq_lens, p.num_seqs, bs,
                       reset_flag ? 1 : 0, flag, tok_off, blk_off, bucket, nb);
    if (remp_status st = hip_check(hipGetLastError(), "expand_scan launch")) return st;
    if (n_desc > 0) {
        const int64_t blocks = (n_desc + 255) / 256;
        hipLaunchKernelGGL(expand_emit, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, stream, dt.seq_lens,
                           dt.row_offsets, dt.block_ids, p.num_seqs, bs, tok_off, blk_off, nnz, num_blocks,
                           p.total_tokens, n_desc, desc, flag, bucket, nb, stamp_at, stamp);
        if (remp_status st = hip_check(hipGetLastError(), "expand_emit launch")) return st;
    }
    return REMP_OK;
}

// Finish the bucket sort of the n_desc new descriptors at desc_off (counted by
// the expansion into bucket_off) into sorted_off; stamp_at receives `stamp`.
static remp_status launch_sort_new(int64_t n_desc, int64_t num_blocks, char* ws, int64_t desc_off,
                                   int64_t bucket_off, int64_t sorted_off, uint64_t* stamp_at, uint64_t stamp,
                                   hipStream_t stream) {
    if (n_desc <= 0) return REMP_OK;
    const uint32_t nb = sort_buckets(n_desc);
    const uint32_t grid = static_cast<uint32_t>((n_desc + 255) / 256);
    const BlockDesc* desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    int32_t* cnt = reinterpret_cast<int32_t*>(ws + bucket_off);
    BlockDesc* out = reinterpret_cast<BlockDesc*>(ws + sorted_off);
    const int64_t nblk = num_blocks > 0 ? num_blocks : 1;
    hipLaunchKernelGGL(sort_scan, dim3(1), dim3(kScanThreads), 0, stream, cnt, nb);
    hipLaunchKernelGGL(sort_scatter, dim3(grid), dim3(256), 0, stream, desc, static_cast<int32_t>(n_desc), nblk, nb,
                       cnt, out, stamp_at, stamp);
    return hip_check(hipGetLastError(), "descriptor sort launch");
}

// Launch shapes measured on MI355X (70B GQA, 7B MHA and DeepSeek-32B shares): small-unit pack runs
// one wave per 4 KiB unit in plain grid order, or four waves of one vector per lane when its units
// are parts of wider rows; everything else takes the XCD-contiguous cell order.
template <int VEC, bool PACK, bool CHECK>
static void launch_copy_vec(const CopyArgs& a, dim3 grid, bool small, bool partial, bool tiny, hipStream_t stream) {
    if (small && PACK && partial)
        hipLaunchKernelGGL((copy_slices<VEC, true, kPackPartialThreads, kPackPartialUnroll, kPackSmallXcd, CHECK>),
                           grid, dim3(kPackPartialThreads), 0, stream, a);
    else if (small && PACK)
        hipLaunchKernelGGL((copy_slices<VEC, true, kPackSmallThreads, kPackSmallUnroll, kPackSmallXcd, CHECK>), grid,
                           dim3(kPackSmallThreads), 0, stream, a);
    else if (small && tiny)
        hipLaunchKernelGGL((copy_slices<VEC, false, kUnpackTinyThreads, kSmallUnroll, kUnpackSmallXcd, CHECK>), grid,
                           dim3(kUnpackTinyThreads), 0, stream, a);
    else if (small)
        hipLaunchKernelGGL((copy_slices<VEC, false, kSmallThreads, kSmallUnroll, kUnpackSmallXcd, CHECK>), grid,
                           dim3(kSmallThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(
            (copy_slices<VEC, PACK, kLargeThreads, kLargeUnroll, PACK ? kPackLargeXcd : kUnpackLargeXcd, CHECK>), grid,
            dim3(kLargeThreads), 0, stream, a);
}

template <int VEC, bool PACK>
static void launch_copy_vec(const CopyArgs& a, dim3 grid, bool small, bool partial, bool tiny, hipStream_t stream) {
    if (a.check.at[0] || a.check.at[1])
        launch_copy_vec<VEC, PACK, true>(a, grid, small, partial, tiny, stream);
    else
        launch_copy_vec<VEC, PACK, false>(a, grid, small, partial, tiny, stream);
}

template <bool PACK>
static remp_status launch_copy(const remp_kv_plan_t& p, const std::vector<HostSlice>& slices, int64_t n_desc,
                               int32_t bs, int64_t block_stride, int32_t row_stride, const char* ws,
                               int64_t desc_off, const StampCheck& check, hipStream_t stream) {
    if (slices.empty() || n_desc == 0) return REMP_OK;
    if (n_desc >= (int64_t(1) << 30)) return fail(REMP_E_UNSUPPORTED, "more than 2^30 live blocks in one call");
    // widest vector every address and stride is aligned to
    uint64_t bits = static_cast<uint64_t>(block_stride) | static_cast<uint64_t>(row_stride) | 16u;
    uint32_t max_row = 0;
    bool partial = false;   // some slice takes only part of each row
    for (const HostSlice& s : slices) {
        bits |= s.paged_k | s.paged_v | s.stage | s.row_bytes |
                (static_cast<uint64_t>(p.total_tokens) * s.row_bytes);
        max_row = std::max(max_row, s.row_bytes);
        partial |= static_cast<int64_t>(s.row_bytes) < row_stride;
    }
    const int vec = static_cast<int>(bits & (~bits + 1));   // lowest set bit, <= 16
    const int64_t per_unit = static_cast<int64_t>(bs) * max_row;
    const bool small = per_unit <= kSmallUnitBytes;
    const int64_t target = wg_target(p, small ? kSmallWgBytes : kLargeWgBytes);
    int32_t C = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(kMaxUnitsPerWg, target / per_unit)));
    // the flattened per-workgroup index stays below 2^31, so a lane's index plus the loop stride
    // (at most 1024 threads x 4 vectors) never wraps in 32 bits
    while (C > 1 && static_cast<uint64_t>(C) * bs * (max_row / vec) >= kMaxWgVectors) C >>= 1;
    if (static_cast<uint64_t>(bs) * (max_row / vec) >= kMaxWgVectors)
        return fail(REMP_E_UNSUPPORTED, "a block of one slice exceeds 2^31 vectors");

    CopyArgs a;
    std::memset(&a, 0, sizeof(a));
    a.desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    a.block_stride = block_stride;
    a.total_tokens = p.total_tokens;
    a.n_desc = static_cast<int32_t>(n_desc);
    a.units_per_wg = C;
    a.row_stride = row_stride;
    a.block_size = bs;
    a.check = check;
    const int64_t gx = (2 * n_desc + C - 1) / C;
    const bool tiny = !PACK && static_cast<int64_t>(C) * per_unit <= kUnpackTinyWgBytes;
    const int threads = small ? (PACK ? (partial ? kPackPartialThreads : kPackSmallThreads)
                                      : (tiny ? kUnpackTinyThreads : kSmallThreads))
                              : kLargeThreads;
    if (remp_status st = check_grid(gx, kMaxItems, threads, PACK ? "pack" : "unpack")) return st;

    if (g_trace_start) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_start, stream), "trace start event")) return st;
    }
    for (size_t first = 0; first < slices.size(); first += kMaxItems) {
        const size_t cnt = std::min<size_t>(kMaxItems, slices.size() - first);
        for (size_t i = 0; i < cnt; ++i) {
            const HostSlice& s = slices[first + i];
            CopyItem& c = a.items[i];
            c.paged_k = s.paged_k;
            c.paged_v = s.paged_v;
            c.stage = s.stage;
            c.row_bytes = s.row_bytes;
            const FastDiv fv = make_fastdiv(s.row_bytes / vec);
            const FastDiv fu = make_fastdiv(static_cast<uint32_t>(bs) * (s.row_bytes / vec));
            c.vpr_magic = fv.magic;
            c.vpr_shift = static_cast<uint16_t>(fv.shift);
            c.unit_magic = fu.magic;
            c.unit_shift = static_cast<uint16_t>(fu.shift);
        }
        const dim3 grid(static_cast<uint32_t>(gx), static_cast<uint32_t>(cnt));
        switch (vec) {
            case 16: launch_copy_vec<16, PACK>(a, grid, small, partial, tiny, stream); break;
            case 8: launch_copy_vec<8, PACK>(a, grid, small, partial, tiny, stream); break;
            case 4: launch_copy_vec<4, PACK>(a, grid, small, partial, tiny, stream); break;
            case 2: launch_copy_vec<2, PACK>(a, grid, small, partial, tiny, stream); break;
            default: launch_copy_vec<1, PACK>(a, grid, small, partial, tiny, stream); break;
        }
        if (remp_status st = hip_check(hipGetLastError(), PACK ? "pack launch" : "unpack launch")) return st;
    }
    if (g_trace_stop) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_stop, stream), "trace stop event")) return st;
    }
    return REMP_OK;
}


template <bool PACK>
static remp_status launch_tiles(const remp_kv_plan_t& p, const std::vector<HostSlice>& slices, int64_t n_desc,
                                int32_t bs, int64_t block_stride, int32_t layout, const char* ws, int64_t desc_off,
                                const StampCheck& check, hipStream_t stream) {
    if (slices.empty() || n_desc == 0) return REMP_OK;
    if (n_desc >= (int64_t(1) << 30)) return fail(REMP_E_UNSUPPORTED, "more than 2^30 live blocks in one call");
    const int32_t eb = p.shape.elem_bytes;
    const int64_t hb = static_cast<int64_t>(p.shape.head_dim) * eb;
    uint64_t bits = static_cast<uint64_t>(block_stride) | static_cast<uint64_t>(hb);
    int32_t max_hc = 1;
    for (const HostSlice& s : slices) {
        bits |= s.paged_k | s.paged_v | s.stage;
        max_hc = std::max<int32_t>(max_hc, static_cast<int32_t>(s.row_bytes / hb));
    }
    if (bits & 15) return fail(REMP_E_ALIGN, "head-tile layouts need 16-byte aligned storage, staging and head rows");
    const int64_t tile_bytes = bs * hb, lrow = hb + 16, tile_lds = bs * lrow;
    if (tile_lds > kTileLdsBytes) return fail(REMP_E_UNSUPPORTED, "a (block, head) tile does not fit in LDS");
    const int32_t tpw = static_cast<int32_t>(std::max<int64_t>(
        1, std::min<int64_t>({kTileWgBytes / tile_bytes, kTileLdsBytes / tile_lds, int64_t(kMaxUnitsPerWg)})));
    const int64_t gx = (n_desc * 2 * max_hc + tpw - 1) / tpw;
    if (remp_status st = check_grid(gx, kMaxItems, kTileThreads, "head tiles")) return st;

    TileArgs a;
    std::memset(&a, 0, sizeof(a));
    a.desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    a.block_stride = block_stride;
    a.total_tokens = p.total_tokens;
    a.n_desc = static_cast<int32_t>(n_desc);
    a.tiles_per_wg = tpw;
    a.block_size = bs;
    a.head_bytes = static_cast<int32_t>(hb);
    a.elem_bytes = eb;
    a.layout = layout;
    a.lds_row = static_cast<int32_t>(lrow);
    const FastDiv fvpt = make_fastdiv(static_cast<uint32_t>(tile_bytes / 16));
    const FastDiv fvph = make_fastdiv(static_cast<uint32_t>(hb / 16));
    const FastDiv fbs = make_fastdiv(static_cast<uint32_t>(bs));
    a.vpt_magic = fvpt.magic;
    a.vpt_shift = fvpt.shift;
    a.vph_magic = fvph.magic;
    a.vph_shift = fvph.shift;
    a.bs_magic = fbs.magic;
    a.bs_shift = fbs.shift;
    a.check = check;
    if (g_trace_start) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_start, stream), "trace start event")) return st;
    }
    for (size_t first = 0; first < slices.size(); first += kMaxItems) {
        const size_t cnt = std::min<size_t>(kMaxItems, slices.size() - first);
        for (size_t i = 0; i < cnt; ++i) {
            const HostSlice& s = slices[first + i];
            a.items[i] = CopyItem{s.paged_k, s.paged_v, s.stage, s.row_bytes, 0, 0, 0, 0};
        }
        const dim3 grid(static_cast<uint32_t>(gx), static_cast<uint32_t>(cnt));
        hipLaunchKernelGGL((copy_tiles<PACK>), grid, dim3(kTileThreads), static_cast<size_t>(tpw * tile_lds), stream, a);
        if (remp_status st = hip_check(hipGetLastError(), PACK ? "pack tile launch" : "unpack tile launch")) return st;
    }
    if (g_trace_stop) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_stop, stream), "trace stop event")) return st;
    }
    return REMP_OK;
}


// Whole paged rows, when every layer of the call splits its rows the same way
// into 2..kMaxMergeSegs staging slices of equal head counts, each share of
// min_seg_bytes..max_seg_bytes, that cover all of the rank's heads.  Returns
// false if not applicable.
template <int VEC, bool PACK>
static void launch_rows_vec(const MergeArgs& a, dim3 grid, bool small, hipStream_t stream) {
    if (small)
        hipLaunchKernelGGL((copy_rows<VEC, PACK, kRowsSmallThreads, kRowsSmallUnroll, false>), grid, dim3(kRowsSmallThreads),
                           0, stream, a);
    else
        hipLaunchKernelGGL((copy_rows<VEC, PACK, kLargeThreads, kLargeUnroll, kRowsLargeXcd>), grid, dim3(kLargeThreads), 0, stream,
                           a);
}

static bool merged_rows_apply(const std::vector<HostSlice>& slices, int32_t heads_per_rank, uint32_t min_seg_bytes,
                              uint32_t max_seg_bytes, std::vector<std::vector<const HostSlice*>>& groups) {
    std::vector<int32_t> layers;
    for (const HostSlice& s : slices)
        if (std::find(layers.begin(), layers.end(), s.layer) == layers.end()) layers.push_back(s.layer);
    groups.clear();
    for (int32_t l : layers) {
        std::vector<const HostSlice*> g;
        for (const HostSlice& s : slices)
            if (s.layer == l) g.push_back(&s);
        std::sort(g.begin(), g.end(), [](const HostSlice* a, const HostSlice* b) { return a->head_local < b->head_local; });
        if (g.size() < 2 || g.size() > static_cast<size_t>(kMaxMergeSegs)) return false;
        int32_t next = 0;                                 // equal slices tile the rank's heads exactly
        for (const HostSlice* s : g) {
            if (s->head_local != next || s->row_bytes < min_seg_bytes || s->row_bytes > max_seg_bytes ||
                s->head_count != g.front()->head_count)
                return false;
            next += s->head_count;
        }
        if (next != heads_per_rank) return false;
        if (!groups.empty()) {                            // same split in every layer
            const auto& f = groups.front();
            for (size_t i = 0; i < g.size(); ++i)
                if (g[i]->head_local != f[i]->head_local || g[i]->head_count != f[i]->head_count) return false;
        }
        groups.push_back(g);
    }
    return !groups.empty();
}

template <bool PACK>
static remp_status launch_rows(const remp_kv_plan_t& p, const std::vector<std::vector<const HostSlice*>>& groups,
                               int64_t n_desc, int32_t bs, int64_t block_stride, int32_t row_stride, const char* ws,
                               int64_t desc_off, const StampCheck& check, hipStream_t stream) {
    if (groups.empty() || n_desc == 0) return REMP_OK;
    // merged_rows_apply admits only equal shares that tile the row: nseg * seg_bytes == row_stride
    const int32_t nseg = static_cast<int32_t>(groups.front().size());
    const uint32_t seg_bytes = groups.front().front()->row_bytes;
    uint64_t bits = static_cast<uint64_t>(block_stride) | static_cast<uint64_t>(row_stride) | seg_bytes | 16u;
    for (const auto& g : groups)
        for (const HostSlice* s : g)
            bits |= s->layer_k | s->layer_v | s->stage | s->row_bytes |
                    (static_cast<uint64_t>(p.total_tokens) * s->row_bytes);
    const int vec = static_cast<int>(bits & (~bits + 1));
    const int64_t per_unit = static_cast<int64_t>(bs) * row_stride;
    const bool small = per_unit <= kSmallUnitBytes;
    const int64_t target = wg_target(p, small ? kSmallWgBytes : kLargeWgBytes);
    int32_t C = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(kMaxUnitsPerWg, target / per_unit)));
    while (C > 1 && static_cast<uint64_t>(C) * bs * (row_stride / vec) >= kMaxWgVectors) C >>= 1;
    if (static_cast<uint64_t>(bs) * (row_stride / vec) >= kMaxWgVectors)
        return fail(REMP_E_UNSUPPORTED, "a block of one row exceeds 2^31 vectors");
    MergeArgs a;
    std::memset(&a, 0, sizeof(a));
    a.desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    a.block_stride = block_stride;
    a.total_tokens = p.total_tokens;
    a.n_desc = static_cast<int32_t>(n_desc);
    a.units_per_wg = C;
    a.row_stride = row_stride;
    a.block_size = bs;
    a.nseg = nseg;
    a.seg_bytes = seg_bytes;
    a.check = check;
    const uint32_t vps = seg_bytes / static_cast<uint32_t>(vec);
    const FastDiv fu = make_fastdiv(static_cast<uint32_t>(bs) * static_cast<uint32_t>(row_stride / vec));
    const FastDiv fs = make_fastdiv(static_cast<uint32_t>(bs) * vps);
    const FastDiv fv = make_fastdiv(vps);
    a.unit_magic = fu.magic;
    a.unit_shift = fu.shift;
    a.seg_magic = fs.magic;
    a.seg_shift = fs.shift;
    a.vps_magic = fv.magic;
    a.vps_shift = fv.shift;
    const int64_t gx = (2 * n_desc + C - 1) / C;
    if (remp_status st = check_grid(gx, kMaxMergeGroups, small ? kRowsSmallThreads : kLargeThreads, "whole rows"))
        return st;
    if (g_trace_start) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_start, stream), "trace start event")) return st;
    }
    for (size_t f = 0; f < groups.size(); f += kMaxMergeGroups) {
        const size_t cnt = std::min<size_t>(kMaxMergeGroups, groups.size() - f);
        for (size_t i = 0; i < cnt; ++i) {
            const auto& g = groups[f + i];
            a.paged_k[i] = g.front()->layer_k;
            a.paged_v[i] = g.front()->layer_v;
            for (size_t k = 0; k < g.size(); ++k) a.stage[i][k] = g[k]->stage;
        }
        const dim3 grid(static_cast<uint32_t>(gx), static_cast<uint32_t>(cnt));
        switch (vec) {
            case 16: launch_rows_vec<16, PACK>(a, grid, small, stream); break;
            case 8: launch_rows_vec<8, PACK>(a, grid, small, stream); break;
            case 4: launch_rows_vec<4, PACK>(a, grid, small, stream); break;
            case 2: launch_rows_vec<2, PACK>(a, grid, small, stream); break;
            default: launch_rows_vec<1, PACK>(a, grid, small, stream); break;
        }
        if (remp_status st = hip_check(hipGetLastError(), PACK ? "pack rows launch" : "unpack rows launch")) return st;
    }
    if (g_trace_stop) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_stop, stream), "trace stop event")) return st;
    }
    return REMP_OK;
}

static bool aligned(const void* p, int64_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

static remp_status check_window(const remp_kv_plan_t* plan, int32_t l0, int32_t l1) {
    if (l0 < 0 || l1 < l0 || l1 > plan->shape.num_layers)
        return fail(REMP_E_RANGE, "layer window [" + std::to_string(l0) + ", " + std::to_string(l1) +
                                      ") outside [0, " + std::to_string(plan->shape.num_layers) + "]");
    return REMP_OK;
}

static remp_status check_pool(const remp_kv_plan_t* plan, const remp_kv_pool* pool, int32_t layers_per_rank,
                              int32_t block_size, const char* what) {
    if (!pool) return fail(REMP_E_INVALID, std::string(what) + " pool is NULL");
    if (pool->layout != kLayoutNHD && pool->layout != kLayoutHND && pool->layout != kLayoutRocmSplit)
        return fail(REMP_E_INVALID, std::string(what) + " pool has an unknown layout");
    const int64_t hb = static_cast<int64_t>(plan->shape.head_dim) * plan->shape.elem_bytes;
    if (pool->layout != kLayoutNHD && hb % 16 != 0)
        return fail(REMP_E_UNSUPPORTED, std::string(what) + " pool layout needs head_dim * elem_bytes % 16 == 0");
    if (pool->layout == kLayoutRocmSplit && (static_cast<int64_t>(block_size) * plan->shape.elem_bytes) % 16 != 0)
        return fail(REMP_E_UNSUPPORTED, std::string(what) + " pool layout needs block_size * elem_bytes % 16 == 0");
    if (pool->num_layers != layers_per_rank)
        return fail(REMP_E_INVALID, std::string(what) + " pool has " + std::to_string(pool->num_layers) +
                                        " layers, the rank holds " + std::to_string(layers_per_rank));
    if (!pool->k || !pool->v) return fail(REMP_E_INVALID, std::string(what) + " pool pointer arrays are NULL");
    return REMP_OK;
}

// A (block, head) tile of block_size rows of head_dim * elem_bytes bytes, each padded by 16 bytes, must fit
// the head-tile kernels' LDS budget; checked with the other arguments, before anything is enqueued.
static remp_status check_tile_fits(const remp_kv_plan_t* plan, int32_t block_size, const char* what) {
    const int64_t hb = static_cast<int64_t>(plan->shape.head_dim) * plan->shape.elem_bytes;
    if (static_cast<int64_t>(block_size) * (hb + 16) > kTileLdsBytes)
        return fail(REMP_E_UNSUPPORTED, std::string(what) + ": a (block, head) tile of " + std::to_string(block_size) +
                                            " rows does not fit the LDS budget of the head-tile kernels");
    return REMP_OK;
}

static remp_status check_workspace(const remp_kv_plan_t* plan, void* ws, int64_t ws_bytes) {
    if (!ws) return fail(REMP_E_INVALID, "workspace is NULL");
    if (!aligned(ws, 256)) return fail(REMP_E_ALIGN, "workspace is not 256-byte aligned");
    if (ws_bytes < workspace_bytes(*plan))
        return fail(REMP_E_SIZE, "workspace has " + std::to_string(ws_bytes) + " bytes, needs " +
                                     std::to_string(workspace_bytes(*plan)));
    return REMP_OK;
}

static remp_status check_dev_tables(const remp_kv_plan_t* plan, const remp_dev_tables* dt, int64_t nnz,
                                    const char* what) {
    if (!dt) return fail(REMP_E_INVALID, std::string("device ") + what + " tables are NULL");
    if (plan->num_seqs > 0 && (!dt->seq_lens || !dt->row_offsets))
        return fail(REMP_E_INVALID, std::string("device ") + what + " table arrays are NULL");
    if (nnz > 0 && !dt->block_ids) return fail(REMP_E_INVALID, std::string("device ") + what + " block ids are NULL");
    return REMP_OK;
}

// New tables describe the planned sequences, every row is long enough, every
// live id is in range and used once, and the pool can hold the live cache.
static remp_status check_new_tables(const remp_kv_plan_t* plan, const remp_block_tables* nt,
                                    const remp_kv_pool* dst, int64_t* nnz_out, uint64_t* stamp_out) {
    if (!nt) return fail(REMP_E_INVALID, "new tables are NULL");
    const remp_block_tables& t = *nt;
    const remp_kv_shape& sh = plan->shape;
    if (t.num_seqs != plan->num_seqs)
        return fail(REMP_E_INVALID, "new tables describe a different number of sequences");
    if (t.num_seqs > 0 && (!t.seq_lens || !t.row_offsets)) return fail(REMP_E_INVALID, "new table arrays are NULL");
    if (t.num_blocks < 0 || t.num_blocks > INT32_MAX) return fail(REMP_E_INVALID, "new num_blocks out of range");
    if (plan->new_live_blocks > t.num_blocks)
        return fail(REMP_E_CAPACITY, "the live cache needs " + std::to_string(plan->new_live_blocks) +
                                         " blocks, the new pool has " + std::to_string(t.num_blocks));
    if (dst->num_blocks < t.num_blocks) return fail(REMP_E_SIZE, "destination pool smaller than its tables");
    int64_t nnz = 0;
    if (t.num_seqs > 0) {
        if (t.row_offsets[0] < 0) return fail(REMP_E_INVALID, "new row_offsets[0] < 0");
        nnz = t.row_offsets[t.num_seqs];
        if (nnz > 0 && !t.block_ids) return fail(REMP_E_INVALID, "new block_ids is NULL");
    }
    std::vector<uint8_t> used(static_cast<size_t>(t.num_blocks), 0);
    // the new descriptors depend on the plan, the pool size (bounds and sort buckets), the table
    // length and the ids the expansion reads
    uint64_t h = mix64(mix64(mix64(mix64(0, plan->serial), 2), static_cast<uint64_t>(t.num_blocks)),
                       static_cast<uint64_t>(nnz));
    for (int32_t q = 0; q < t.num_seqs; ++q) {
        if (t.seq_lens[q] != plan->seq_lens[q])
            return fail(REMP_E_INVALID, "new tables give sequence " + std::to_string(q) + " length " +
                                            std::to_string(t.seq_lens[q]) + ", planned " +
                                            std::to_string(plan->seq_lens[q]));
        const int32_t a = t.row_offsets[q], b = t.row_offsets[q + 1];
        if (b < a) return fail(REMP_E_INVALID, "new row_offsets decrease at sequence " + std::to_string(q));
        const int64_t need = ceil_div(t.seq_lens[q], sh.new_block_size);
        if (b - a < need) return fail(REMP_E_INVALID, "new table row of sequence " + std::to_string(q) + " too short");
        h = mix64(h, static_cast<uint32_t>(a));
        for (int64_t j = 0; j < need; ++j) {
            const int32_t id = t.block_ids[a + j];
            if (id < 0 || id >= t.num_blocks)
                return fail(REMP_E_RANGE, "new block id " + std::to_string(id) + " outside [0, " +
                                              std::to_string(t.num_blocks) + ")");
            if (used[id]) return fail(REMP_E_INVALID, "new block id " + std::to_string(id) + " used twice");
            used[id] = 1;
            h = mix64(h, static_cast<uint32_t>(id));
        }
    }
    *nnz_out = nnz;
    *stamp_out = finish64(h);
    return REMP_OK;
}

// Slices of the window for one side; fills `out`.  `pack`: items of old rank
// `rank`; else items of new rank `rank`.  skip_local leaves out the slices
// whose peer is the same global rank.
static remp_status collect_slices(const remp_kv_plan_t& p, bool pack, int32_t rank, int32_t l0, int32_t l1,
                                  const remp_kv_pool& pool, const remp_buffer* staging, bool skip_local,
                                  std::vector<HostSlice>& out) {
    const Ownership& mine = pack ? p.own_old : p.own_new;
    const int64_t hrow = static_cast<int64_t>(p.shape.head_dim) * p.shape.elem_bytes;
    const int32_t eb = p.shape.elem_bytes;
    for (const Item& it : p.items) {
        if ((pack ? it.src : it.dst) != rank || it.layer < l0 || it.layer >= l1) continue;
        const int32_t peer = pack ? it.dst : it.src;
        if (skip_local && peer == rank) continue;
        const Pair& pr = p.pairs[it.pair];
        const int32_t ws0 = std::max(l0, pr.layer_begin), ws1 = std::min(l1, pr.layer_end);
        const remp_buffer& sb = staging[peer];
        const int64_t need = static_cast<int64_t>(ws1 - ws0) * pr.slice_bytes;
        if (need > 0) {
            if (!sb.ptr)
                return fail(REMP_E_INVALID, std::string("staging buffer for ") + (pack ? "destination " : "source ") +
                                                std::to_string(peer) + " is NULL");
            if (sb.bytes < need)
                return fail(REMP_E_SIZE, "staging buffer for rank " + std::to_string(peer) + " has " +
                                             std::to_string(sb.bytes) + " bytes, the window needs " +
                                             std::to_string(need));
            if (!aligned(sb.ptr, eb)) return fail(REMP_E_ALIGN, "staging buffer not element aligned");
        }
        const int32_t li = it.layer - mine.first_layer(rank);
        void* k = pool.k[li];
        void* v = pool.v[li];
        if (!k || !v)
            return fail(REMP_E_INVALID, "pool storage of layer " + std::to_string(it.layer) + " is NULL");
        if (!aligned(k, eb) || !aligned(v, eb)) return fail(REMP_E_ALIGN, "pool storage not element aligned");
        const int64_t hstep = pool.layout == kLayoutNHD
                                  ? hrow
                                  : hrow * (pack ? p.shape.old_block_size : p.shape.new_block_size);
        const int64_t hoff = static_cast<int64_t>(it.head_begin - mine.first_head(rank)) * hstep;
        HostSlice s;
        s.paged_k = reinterpret_cast<uint64_t>(k) + hoff;
        s.paged_v = reinterpret_cast<uint64_t>(v) + hoff;
        s.stage = reinterpret_cast<uint64_t>(sb.ptr) + static_cast<uint64_t>(it.layer - ws0) * pr.slice_bytes;
        s.row_bytes = static_cast<uint32_t>(it.head_count * hrow);
        s.layer = it.layer;
        s.head_local = it.head_begin - mine.first_head(rank);
        s.head_count = it.head_count;
        s.layer_k = reinterpret_cast<uint64_t>(k);
        s.layer_v = reinterpret_cast<uint64_t>(v);
        out.push_back(s);
    }
    return REMP_OK;
}

// In an HND pool the rows of one head's tile are contiguous and in token
// order, so a slice of a single head has the staging slice's byte order: it is
// copied like an NHD slice whose rows are one head long.  Used for pack (A/B
// on MI355X, 70B GQA share with HND pools: pack -4.3% time against the LDS
// tile kernel); the unpack keeps the tile kernel (+1.2% with the direct copy).
static bool hnd_single_heads(int32_t layout, const std::vector<HostSlice>& slices) {
    if (layout != kLayoutHND) return false;
    for (const HostSlice& s : slices)
        if (s.head_count != 1) return false;
    return true;
}

// ---------------------------------------------------------------------------
// local copy: old pool -> new pool for slices that stay on the same rank
// ---------------------------------------------------------------------------

struct HostLocal {
    uint64_t src_k, src_v, dst_k, dst_v;
    uint32_t row_bytes;
};

template <int VEC>
static remp_status launch_local_vec(const LocalArgs& a, dim3 grid, bool small, hipStream_t stream) {
    if (small)
        hipLaunchKernelGGL((copy_local<VEC, kLocalSmallThreads, kLocalSmallUnroll, false>), grid, dim3(kLocalSmallThreads), 0,
                           stream, a);
    else
        hipLaunchKernelGGL((copy_local<VEC, kLocalLargeThreads, kLocalLargeUnroll, kLocalLargeXcd>), grid, dim3(kLocalLargeThreads), 0,
                           stream, a);
    return hip_check(hipGetLastError(), "copy_local launch");
}

// Local copy when either pool is not NHD: head tiles through LDS.  items carry
// the slice's first-head offsets in each pool's own layout.
static remp_status launch_local_tiles(const remp_kv_plan_t& p, const std::vector<HostLocal>& items,
                                      int32_t old_layout, int32_t new_layout, const char* ws,
                                      const StampCheck& check, hipStream_t stream) {
    const remp_kv_shape& sh = p.shape;
    const WorkspaceLayout L = workspace_layout(p);
    const int64_t n_desc = p.new_live_blocks;
    if (items.empty() || n_desc == 0) return REMP_OK;
    if (n_desc >= (int64_t(1) << 28)) return fail(REMP_E_UNSUPPORTED, "more than 2^28 live blocks in one call");
    const int32_t eb = sh.elem_bytes;
    const int64_t hb = static_cast<int64_t>(sh.head_dim) * eb;
    if (hb % 16 != 0) return fail(REMP_E_UNSUPPORTED, "head tiles need head_dim * elem_bytes % 16 == 0");
    const int32_t bo = sh.old_block_size, bn = sh.new_block_size;
    if (bn > kMaxLocalRows) return fail(REMP_E_UNSUPPORTED, "new block size above the local-copy row limit");
    const int64_t lds_row = hb + 16;
    const int64_t tile_lds = bn * lds_row;
    if (tile_lds > kTileLdsBytes) return fail(REMP_E_UNSUPPORTED, "a head tile does not fit the LDS budget");
    int64_t T = std::max<int64_t>(1, kTileWgBytes / (bn * hb));
    T = std::min<int64_t>({T, kTileLdsBytes / tile_lds, kMaxLocalRows / bn, kMaxUnitsPerWg});
    const int64_t orow = p.own_old.heads_per_rank() * hb, nrow = p.own_new.heads_per_rank() * hb;

    LocalTileArgs a;
    std::memset(&a, 0, sizeof(a));
    a.new_desc = reinterpret_cast<const BlockDesc*>(ws + L.sorted_new);
    a.old_desc = reinterpret_cast<const BlockDesc*>(ws + L.desc_old);
    a.tok_off = reinterpret_cast<const int32_t*>(ws + L.scan_old);
    a.old_blk_off = reinterpret_cast<const int32_t*>(ws + L.scan_old) + (p.num_seqs + 1);
    a.flag = reinterpret_cast<int32_t*>(const_cast<char*>(ws));
    a.old_block_stride = orow * bo;
    a.new_block_stride = nrow * bn;
    a.n_new_desc = static_cast<int32_t>(n_desc);
    a.n_old_desc = static_cast<int32_t>(p.old_live_blocks);
    a.tiles_per_wg = static_cast<int32_t>(T);
    a.old_block_size = bo;
    a.new_block_size = bn;
    a.head_bytes = static_cast<int32_t>(hb);
    a.elem_bytes = eb;
    a.old_layout = old_layout;
    a.new_layout = new_layout;
    a.old_row_stride = static_cast<int32_t>(orow);
    a.new_row_stride = static_cast<int32_t>(nrow);
    a.old_head_step = static_cast<int32_t>(old_layout == kLayoutNHD ? hb : hb * bo);
    a.new_head_step = static_cast<int32_t>(new_layout == kLayoutNHD ? hb : hb * bn);
    a.lds_row = static_cast<int32_t>(lds_row);
    const FastDiv fv = make_fastdiv(static_cast<uint32_t>(hb / 16));
    const FastDiv fr = make_fastdiv(static_cast<uint32_t>(bn * (hb / 16)));
    const FastDiv fb = make_fastdiv(static_cast<uint32_t>(bn));
    a.vph_magic = fv.magic;
    a.vph_shift = fv.shift;
    a.rows_magic = fr.magic;
    a.rows_shift = fr.shift;
    a.bn_magic = fb.magic;
    a.bn_shift = fb.shift;
    a.check = check;
    if (g_trace_start) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_start, stream), "trace start event")) return st;
    }
    for (size_t first = 0; first < items.size(); first += kMaxLocalTileItems) {
        const size_t cnt = std::min<size_t>(kMaxLocalTileItems, items.size() - first);
        int32_t max_hc = 1;
        for (size_t i = 0; i < cnt; ++i) {
            const HostLocal& h = items[first + i];
            LocalTileItem& c = a.items[i];
            c.src_k = h.src_k;
            c.src_v = h.src_v;
            c.dst_k = h.dst_k;
            c.dst_v = h.dst_v;
            c.heads = static_cast<int32_t>(h.row_bytes / hb);
            max_hc = std::max(max_hc, c.heads);
        }
        const int64_t gx = (n_desc * 2 * max_hc + T - 1) / T;
        if (remp_status st = check_grid(gx, kMaxLocalTileItems, kTileThreads, "local head tiles")) return st;
        // 32-bit vector indices per workgroup: T tiles of bn rows of hb / 16 vectors
        hipLaunchKernelGGL(copy_local_tiles, dim3(static_cast<uint32_t>(gx), static_cast<uint32_t>(cnt)),
                           dim3(kTileThreads), static_cast<size_t>(local_tile_lds_bytes(T, bn, lds_row)), stream, a);
        if (remp_status st = hip_check(hipGetLastError(), "copy_local_tiles launch")) return st;
    }
    if (g_trace_stop) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_stop, stream), "trace stop event")) return st;
    }
    return REMP_OK;
}

static remp_status launch_local(const remp_kv_plan_t& p, const std::vector<HostLocal>& items, const char* ws,
                                const StampCheck& check, hipStream_t stream) {
    const remp_kv_shape& sh = p.shape;
    const WorkspaceLayout L = workspace_layout(p);
    const int64_t n_desc = p.new_live_blocks;
    if (items.empty() || n_desc == 0) return REMP_OK;
    if (n_desc >= (int64_t(1) << 30)) return fail(REMP_E_UNSUPPORTED, "more than 2^30 live blocks in one call");
    const int64_t hrow = static_cast<int64_t>(sh.head_dim) * sh.elem_bytes;
    const int64_t orow = p.own_old.heads_per_rank() * hrow, nrow = p.own_new.heads_per_rank() * hrow;
    const int32_t bo = sh.old_block_size, bn = sh.new_block_size;
    uint64_t bits = static_cast<uint64_t>(orow) | static_cast<uint64_t>(nrow) | 16u;
    uint32_t max_row = 0;
    for (const HostLocal& it : items) {
        bits |= it.src_k | it.src_v | it.dst_k | it.dst_v | it.row_bytes;
        max_row = std::max(max_row, it.row_bytes);
    }
    const int vec = static_cast<int>(bits & (~bits + 1));
    const int64_t per_unit = static_cast<int64_t>(bn) * max_row;
    const bool small = per_unit <= kSmallUnitBytes;
    const int64_t target = wg_target(p, small ? kLocalSmallWgBytes : kLocalLargeWgBytes);
    int32_t C = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(kMaxUnitsPerWg, target / per_unit)));
    C = std::min<int32_t>(C, std::max<int32_t>(1, kMaxLocalRows / bn));
    if (bn > kMaxLocalRows) return fail(REMP_E_UNSUPPORTED, "new block size above the local-copy row limit");
    while (C > 1 && static_cast<uint64_t>(C) * bn * (max_row / vec) >= kMaxWgVectors) C >>= 1;
    if (static_cast<uint64_t>(bn) * (max_row / vec) >= kMaxWgVectors)
        return fail(REMP_E_UNSUPPORTED, "a block of one slice exceeds 2^31 vectors");

    LocalArgs a;
    std::memset(&a, 0, sizeof(a));
    a.new_desc = reinterpret_cast<const BlockDesc*>(ws + L.sorted_new);
    a.old_desc = reinterpret_cast<const BlockDesc*>(ws + L.desc_old);
    a.tok_off = reinterpret_cast<const int32_t*>(ws + L.scan_old);
    a.old_blk_off = reinterpret_cast<const int32_t*>(ws + L.scan_old) + (p.num_seqs + 1);
    a.flag = reinterpret_cast<int32_t*>(const_cast<char*>(ws));
    a.old_block_stride = orow * bo;
    a.new_block_stride = nrow * bn;
    a.n_new_desc = static_cast<int32_t>(n_desc);
    a.n_old_desc = static_cast<int32_t>(p.old_live_blocks);
    a.units_per_wg = C;
    a.old_row_stride = static_cast<int32_t>(orow);
    a.new_row_stride = static_cast<int32_t>(nrow);
    a.old_block_size = bo;
    a.new_block_size = bn;
    a.check = check;
    const int64_t gx = (2 * n_desc + C - 1) / C;
    if (remp_status st = check_grid(gx, kMaxLocalItems, small ? kLocalSmallThreads : kLocalLargeThreads, "local copy"))
        return st;
    if (g_trace_start) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_start, stream), "trace start event")) return st;
    }
    for (size_t first = 0; first < items.size(); first += kMaxLocalItems) {
        const size_t cnt = std::min<size_t>(kMaxLocalItems, items.size() - first);
        for (size_t i = 0; i < cnt; ++i) {
            const HostLocal& h = items[first + i];
            LocalItem& c = a.items[i];
            c.src_k = h.src_k;
            c.src_v = h.src_v;
            c.dst_k = h.dst_k;
            c.dst_v = h.dst_v;
            c.row_bytes = h.row_bytes;
            const FastDiv fv = make_fastdiv(h.row_bytes / vec);
            const FastDiv fu = make_fastdiv(static_cast<uint32_t>(bn) * (h.row_bytes / vec));
            c.vpr_magic = fv.magic;
            c.vpr_shift = static_cast<uint16_t>(fv.shift);
            c.unit_magic = fu.magic;
            c.unit_shift = static_cast<uint16_t>(fu.shift);
        }
        const dim3 grid(static_cast<uint32_t>(gx), static_cast<uint32_t>(cnt));
        remp_status st;
        switch (vec) {
            case 16: st = launch_local_vec<16>(a, grid, small, stream); break;
            case 8: st = launch_local_vec<8>(a, grid, small, stream); break;
            case 4: st = launch_local_vec<4>(a, grid, small, stream); break;
            case 2: st = launch_local_vec<2>(a, grid, small, stream); break;
            default: st = launch_local_vec<1>(a, grid, small, stream); break;
        }
        if (st) return st;
    }
    if (g_trace_stop) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_stop, stream), "trace stop event")) return st;
    }
    return REMP_OK;
}

static bool ranges_overlap(uint64_t a, uint64_t an, uint64_t b, uint64_t bn) { return a < b + bn && b < a + an; }

// Argument checks shared by the unpack entry points (everything but the workspace and the tables).
static remp_status check_unpack_args(const remp_kv_plan_t* plan, int32_t new_rank, int32_t layer_begin,
                                     int32_t layer_end, const remp_buffer* staging, const remp_kv_pool* dst,
                                     uint32_t flags) {
    if (flags & ~static_cast<uint32_t>(REMP_KV_SKIP_LOCAL | REMP_KV_REUSE_DESCRIPTORS))
        return fail(REMP_E_INVALID, "unknown flags");
    if (new_rank < 0 || new_rank >= plan->own_new.world())
        return fail(REMP_E_RANGE, "new_rank " + std::to_string(new_rank) + " outside [0, " +
                                      std::to_string(plan->own_new.world()) + ")");
    if (remp_status st = check_window(plan, layer_begin, layer_end)) return st;
    if (remp_status st = check_pool(plan, dst, plan->own_new.layers_of_rank(new_rank), plan->shape.new_block_size,
                                    "destination"))
        return st;
    if (!staging) return fail(REMP_E_INVALID, "staging array is NULL");
    return REMP_OK;
}

// Unpack with its scratch areas at `ws` (laid out by workspace_layout) and the status flag at `flag`.
static remp_status unpack_impl(const remp_kv_plan_t* plan, int32_t new_rank, int32_t layer_begin, int32_t layer_end,
                               const remp_buffer* staging, const remp_kv_pool* dst,
                               const remp_block_tables* new_tables, const remp_dev_tables* new_dev_tables, char* ws,
                               int32_t* flag, uint32_t flags, hipStream_t stream) {
    int64_t nnz = 0;
    uint64_t new_stamp = 0;
    if (remp_status st = check_new_tables(plan, new_tables, dst, &nnz, &new_stamp)) return st;
    if (remp_status st = check_dev_tables(plan, new_dev_tables, nnz, "new")) return st;

    std::vector<HostSlice> slices;
    if (remp_status st = collect_slices(*plan, false, new_rank, layer_begin, layer_end, *dst, staging,
                                        (flags & REMP_KV_SKIP_LOCAL) != 0, slices))
        return st;
    if (dst->layout != kLayoutNHD)
        if (remp_status st = check_tile_fits(plan, plan->shape.new_block_size, "unpack")) return st;
    if (layer_begin == layer_end || plan->new_live_blocks == 0) return REMP_OK;   // as in pack
    const remp_kv_shape& sh = plan->shape;
    const int64_t row_stride = static_cast<int64_t>(plan->own_new.heads_per_rank()) * sh.head_dim * sh.elem_bytes;
    const WorkspaceLayout L = workspace_layout(*plan);
    uint64_t* new_at = reinterpret_cast<uint64_t*>(ws + L.stamp_new);
    StampCheck check = no_check(flag);
    if (flags & REMP_KV_REUSE_DESCRIPTORS) {
        check.at[0] = new_at;
        check.want[0] = new_stamp;
    } else {
        if (remp_status st = launch_expand(*plan, *new_dev_tables, sh.new_block_size, nnz, new_tables->num_blocks,
                                           plan->new_live_blocks, ws, flag, L.scan_new, L.desc_new, true, stream,
                                           L.bucket_new, nullptr, 0))
            return st;
        if (remp_status st = launch_sort_new(plan->new_live_blocks, new_tables->num_blocks, ws, L.desc_new,
                                             L.bucket_new, L.sorted_new, new_at, new_stamp, stream))
            return st;
    }
    if (dst->layout != kLayoutNHD)
        return launch_tiles<false>(*plan, slices, plan->new_live_blocks, sh.new_block_size,
                                   row_stride * sh.new_block_size, dst->layout, ws, L.sorted_new, check, stream);
    std::vector<std::vector<const HostSlice*>> groups;
    if (kMergeRows && merged_rows_apply(slices, plan->own_new.heads_per_rank(), kUnpackRowsMinShareBytes,
                                        kUnpackRowsMaxShareBytes, groups))
        return launch_rows<false>(*plan, groups, plan->new_live_blocks, sh.new_block_size, row_stride * sh.new_block_size,
                           static_cast<int32_t>(row_stride), ws, L.sorted_new, check, stream);
    return launch_copy<false>(*plan, slices, plan->new_live_blocks, sh.new_block_size, row_stride * sh.new_block_size,
                              static_cast<int32_t>(row_stride), ws, L.sorted_new, check, stream);
}

// ---------------------------------------------------------------------------
// static scratch of the allocation-free unpack
// ---------------------------------------------------------------------------
//
// remp_kv_unpack_noalloc keeps its workspace areas in this array instead of a
// caller buffer.  Each device that loads the library holds its own copy until
// the process ends; the host-side name below is only a stand-in, so kernels
// get the device address that hipGetSymbolAddress returns for the current
// device, resolved once per device on that device's first call.
constexpr int64_t kScratchBytes = REMP_KV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
static std::atomic<char*> g_scratch_ptr[kMaxScratchDevices];
static std::mutex g_scratch_mu;

static remp_status scratch_of_current_device(hipStream_t stream, char** out) {
    int dev = -1;
    if (remp_status st = hip_check(hipGetDevice(&dev), "hipGetDevice")) return st;
    if (stream) {   // the kernels run on the stream's device: its scratch must be that device's copy
        hipDevice_t sdev = -1;
        if (remp_status st = hip_check(hipStreamGetDevice(stream, &sdev), "hipStreamGetDevice")) return st;
        if (sdev != dev)
            return fail(REMP_E_INVALID, "the stream belongs to device " + std::to_string(sdev) +
                                            ", the current device is " + std::to_string(dev));
    }
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(REMP_E_UNSUPPORTED, "device index " + std::to_string(dev) + " beyond the static scratch table");
    char* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            void* addr = nullptr;
            if (remp_status st = hip_check(hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)),
                                           "hipGetSymbolAddress(scratch)"))
                return st;
            if (!addr || !aligned(addr, 256)) return fail(REMP_E_HIP, "static scratch has no 256-byte aligned address");
            p = static_cast<char*>(addr);
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return REMP_OK;
}

}  // namespace remp

using namespace remp;

extern "C" {

void remp_kv_set_trace_events(hipEvent_t start, hipEvent_t stop) {
    g_trace_start = start;
    g_trace_stop = stop;
}

remp_status remp_kv_pack(const remp_kv_plan_t* plan, int32_t old_rank, int32_t layer_begin, int32_t layer_end,
                         const remp_kv_pool* src, const remp_dev_tables* old_tables, const remp_buffer* staging,
                         void* workspace, int64_t workspace_bytes_, uint32_t flags, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    if (flags & ~static_cast<uint32_t>(REMP_KV_SKIP_LOCAL | REMP_KV_REUSE_DESCRIPTORS))
        return fail(REMP_E_INVALID, "unknown flags");
    if (old_rank < 0 || old_rank >= plan->own_old.world())
        return fail(REMP_E_RANGE, "old_rank " + std::to_string(old_rank) + " outside [0, " +
                                      std::to_string(plan->own_old.world()) + ")");
    if (remp_status st = check_window(plan, layer_begin, layer_end)) return st;
    if (remp_status st = check_pool(plan, src, plan->own_old.layers_of_rank(old_rank), plan->shape.old_block_size,
                                    "source"))
        return st;
    if (!staging) return fail(REMP_E_INVALID, "staging array is NULL");
    if (remp_status st = check_workspace(plan, workspace, workspace_bytes_)) return st;
    if (src->num_blocks < plan->old_num_blocks)
        return fail(REMP_E_SIZE, "source pool has fewer blocks than the old tables address");
    if (remp_status st = check_dev_tables(plan, old_tables, plan->old_nnz, "old")) return st;

    std::vector<HostSlice> slices;
    if (remp_status st = collect_slices(*plan, true, old_rank, layer_begin, layer_end, *src, staging,
                                        (flags & REMP_KV_SKIP_LOCAL) != 0, slices))
        return st;
    if (src->layout != kLayoutNHD && !hnd_single_heads(src->layout, slices))
        if (remp_status st = check_tile_fits(plan, plan->shape.old_block_size, "pack")) return st;
    // an empty window or cache does nothing; otherwise the tables are expanded (and their stamp
    // written) even when the rank has no slice in the window, so that later calls may reuse them
    if (layer_begin == layer_end || plan->old_live_blocks == 0) return REMP_OK;
    const remp_kv_shape& sh = plan->shape;
    const int64_t row_stride = static_cast<int64_t>(plan->own_old.heads_per_rank()) * sh.head_dim * sh.elem_bytes;
    const WorkspaceLayout L = workspace_layout(*plan);
    char* ws = static_cast<char*>(workspace);
    uint64_t* old_at = reinterpret_cast<uint64_t*>(ws + L.stamp_old);
    int32_t* flag = reinterpret_cast<int32_t*>(ws);
    StampCheck check = no_check(flag);
    if (flags & REMP_KV_REUSE_DESCRIPTORS) {
        check.at[0] = old_at;
        check.want[0] = old_stamp(*plan);
    } else if (remp_status st = launch_expand(*plan, *old_tables, sh.old_block_size, plan->old_nnz,
                                              plan->old_num_blocks, plan->old_live_blocks, ws, flag, L.scan_old,
                                              L.desc_old, true, stream, -1, old_at, old_stamp(*plan))) {
        return st;
    }
    if (hnd_single_heads(src->layout, slices))
        return launch_copy<true>(*plan, slices, plan->old_live_blocks, sh.old_block_size,
                                 row_stride * sh.old_block_size,
                                 static_cast<int32_t>(row_stride / plan->own_old.heads_per_rank()), ws, L.desc_old,
                                 check, stream);
    if (src->layout != kLayoutNHD)
        return launch_tiles<true>(*plan, slices, plan->old_live_blocks, sh.old_block_size,
                                  row_stride * sh.old_block_size, src->layout, ws, L.desc_old, check, stream);
    std::vector<std::vector<const HostSlice*>> groups;
    if (kPackRows && merged_rows_apply(slices, plan->own_old.heads_per_rank(), kPackRowsMinShareBytes,
                                       kPackRowsMaxShareBytes, groups))
        return launch_rows<true>(*plan, groups, plan->old_live_blocks, sh.old_block_size,
                                 row_stride * sh.old_block_size, static_cast<int32_t>(row_stride), ws, L.desc_old, check,
                                 stream);
    return launch_copy<true>(*plan, slices, plan->old_live_blocks, sh.old_block_size, row_stride * sh.old_block_size,
                             static_cast<int32_t>(row_stride), ws, L.desc_old, check, stream);
}

remp_status remp_kv_unpack(const remp_kv_plan_t* plan, int32_t new_rank, int32_t layer_begin, int32_t layer_end,
                           const remp_buffer* staging, const remp_kv_pool* dst, const remp_block_tables* new_tables,
                           const remp_dev_tables* new_dev_tables, void* workspace, int64_t workspace_bytes_,
                           uint32_t flags, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    if (remp_status st = check_unpack_args(plan, new_rank, layer_begin, layer_end, staging, dst, flags)) return st;
    if (remp_status st = check_workspace(plan, workspace, workspace_bytes_)) return st;
    char* ws = static_cast<char*>(workspace);
    return unpack_impl(plan, new_rank, layer_begin, layer_end, staging, dst, new_tables, new_dev_tables, ws,
                       reinterpret_cast<int32_t*>(ws), flags, stream);
}

remp_status remp_kv_unpack_noalloc(const remp_kv_plan_t* plan, int32_t new_rank, int32_t layer_begin,
                                   int32_t layer_end, const remp_buffer* staging, const remp_kv_pool* dst,
                                   const remp_block_tables* new_tables, const remp_dev_tables* new_dev_tables,
                                   int32_t* status, uint32_t flags, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    if (workspace_bytes(*plan) > kScratchBytes)
        return fail(REMP_E_SIZE, "the plan needs " + std::to_string(workspace_bytes(*plan)) +
                                     " bytes of scratch, the static scratch holds " + std::to_string(kScratchBytes));
    if (status && !aligned(status, 4)) return fail(REMP_E_ALIGN, "status is not 4-byte aligned");
    if (remp_status st = check_unpack_args(plan, new_rank, layer_begin, layer_end, staging, dst, flags)) return st;
    char* ws = nullptr;
    if (remp_status st = scratch_of_current_device(stream, &ws)) return st;
    return unpack_impl(plan, new_rank, layer_begin, layer_end, staging, dst, new_tables, new_dev_tables, ws,
                       status ? status : reinterpret_cast<int32_t*>(ws), flags, stream);
}

remp_status remp_kv_copy_local(const remp_kv_plan_t* plan, int32_t rank, int32_t layer_begin, int32_t layer_end,
                               const remp_kv_pool* src, const remp_dev_tables* old_tables, const remp_kv_pool* dst,
                               const remp_block_tables* new_tables, const remp_dev_tables* new_dev_tables,
                               void* workspace, int64_t workspace_bytes_, uint32_t flags, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    if (flags & ~static_cast<uint32_t>(REMP_KV_REUSE_DESCRIPTORS)) return fail(REMP_E_INVALID, "unknown flags");
    if (rank < 0 || rank >= plan->own_old.world() || rank >= plan->own_new.world())
        return fail(REMP_E_RANGE, "rank " + std::to_string(rank) + " is not a rank of both topologies");
    if (remp_status st = check_window(plan, layer_begin, layer_end)) return st;
    if (remp_status st = check_pool(plan, src, plan->own_old.layers_of_rank(rank), plan->shape.old_block_size,
                                    "source"))
        return st;
    if (remp_status st = check_pool(plan, dst, plan->own_new.layers_of_rank(rank), plan->shape.new_block_size,
                                    "destination"))
        return st;
    if (remp_status st = check_workspace(plan, workspace, workspace_bytes_)) return st;
    if (src->num_blocks < plan->old_num_blocks)
        return fail(REMP_E_SIZE, "source pool has fewer blocks than the old tables address");
    if (remp_status st = check_dev_tables(plan, old_tables, plan->old_nnz, "old")) return st;
    int64_t nnz = 0;
    uint64_t new_stamp = 0;
    if (remp_status st = check_new_tables(plan, new_tables, dst, &nnz, &new_stamp)) return st;
    if (remp_status st = check_dev_tables(plan, new_dev_tables, nnz, "new")) return st;

    const remp_kv_shape& sh = plan->shape;
    const int64_t hrow = static_cast<int64_t>(sh.head_dim) * sh.elem_bytes;
    const int64_t old_layer_bytes = plan->own_old.heads_per_rank() * hrow * sh.old_block_size * src->num_blocks;
    const int64_t new_layer_bytes = plan->own_new.heads_per_rank() * hrow * sh.new_block_size * dst->num_blocks;
    const int32_t eb = sh.elem_bytes;
    std::vector<HostLocal> items;
    for (const Item& it : plan->items) {
        if (it.src != rank || it.dst != rank || it.layer < layer_begin || it.layer >= layer_end) continue;
        const int32_t lo = it.layer - plan->own_old.first_layer(rank), ln = it.layer - plan->own_new.first_layer(rank);
        void* sk = src->k[lo];
        void* sv = src->v[lo];
        void* dk = dst->k[ln];
        void* dv = dst->v[ln];
        if (!sk || !sv || !dk || !dv)
            return fail(REMP_E_INVALID, "pool storage of layer " + std::to_string(it.layer) + " is NULL");
        if (!aligned(sk, eb) || !aligned(sv, eb) || !aligned(dk, eb) || !aligned(dv, eb))
            return fail(REMP_E_ALIGN, "pool storage not element aligned");
        const uint64_t s2[2] = {reinterpret_cast<uint64_t>(sk), reinterpret_cast<uint64_t>(sv)};
        const uint64_t d2[2] = {reinterpret_cast<uint64_t>(dk), reinterpret_cast<uint64_t>(dv)};
        for (uint64_t a : s2)
            for (uint64_t b : d2)
                if (ranges_overlap(a, old_layer_bytes, b, new_layer_bytes))
                    return fail(REMP_E_INVALID, "old and new storage of layer " + std::to_string(it.layer) + " overlap");
        // offset of the slice's first head: a row run in NHD, a whole head tile in the tile layouts
        const uint64_t ostep = src->layout == kLayoutNHD ? hrow : hrow * sh.old_block_size;
        const uint64_t nstep = dst->layout == kLayoutNHD ? hrow : hrow * sh.new_block_size;
        HostLocal h;
        h.src_k = s2[0] + static_cast<uint64_t>(it.head_begin - plan->own_old.first_head(rank)) * ostep;
        h.src_v = s2[1] + static_cast<uint64_t>(it.head_begin - plan->own_old.first_head(rank)) * ostep;
        h.dst_k = d2[0] + static_cast<uint64_t>(it.head_begin - plan->own_new.first_head(rank)) * nstep;
        h.dst_v = d2[1] + static_cast<uint64_t>(it.head_begin - plan->own_new.first_head(rank)) * nstep;
        h.row_bytes = static_cast<uint32_t>(it.head_count * hrow);
        items.push_back(h);
    }
    if (src->layout != kLayoutNHD || dst->layout != kLayoutNHD) {
        if (remp_status st = check_tile_fits(plan, sh.new_block_size, "local copy")) return st;
    }
    if (sh.new_block_size > kMaxLocalRows)
        return fail(REMP_E_UNSUPPORTED, "new block size above the local-copy row limit");
    if (layer_begin == layer_end || plan->new_live_blocks == 0) return REMP_OK;   // as in pack
    const WorkspaceLayout L = workspace_layout(*plan);
    char* ws = static_cast<char*>(workspace);
    uint64_t* old_at = reinterpret_cast<uint64_t*>(ws + L.stamp_old);
    uint64_t* new_at = reinterpret_cast<uint64_t*>(ws + L.stamp_new);
    int32_t* flag = reinterpret_cast<int32_t*>(ws);
    StampCheck check = no_check(flag);
    if (flags & REMP_KV_REUSE_DESCRIPTORS) {
        check.at[0] = old_at;
        check.want[0] = old_stamp(*plan);
        check.at[1] = new_at;
        check.want[1] = new_stamp;
    } else {
        if (remp_status st = launch_expand(*plan, *old_tables, sh.old_block_size, plan->old_nnz,
                                           plan->old_num_blocks, plan->old_live_blocks, ws, flag, L.scan_old,
                                           L.desc_old, true, stream, -1, old_at, old_stamp(*plan)))
            return st;
        if (remp_status st = launch_expand(*plan, *new_dev_tables, sh.new_block_size, nnz, new_tables->num_blocks,
                                           plan->new_live_blocks, ws, flag, L.scan_new, L.desc_new, false, stream,
                                           L.bucket_new, nullptr, 0))
            return st;
        if (remp_status st = launch_sort_new(plan->new_live_blocks, new_tables->num_blocks, ws, L.desc_new,
                                             L.bucket_new, L.sorted_new, new_at, new_stamp, stream))
            return st;
    }
    if (src->layout != kLayoutNHD || dst->layout != kLayoutNHD)
        return launch_local_tiles(*plan, items, src->layout, dst->layout, ws, check, stream);
    return launch_local(*plan, items, ws, check, stream);
}

}  // extern "C"
