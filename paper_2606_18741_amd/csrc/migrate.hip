// GPU side of the KV-cache migration for gfx950: block-table expansion and the
// pack / unpack copy kernels, plus the two C entry points that launch them.
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
#include <cstdlib>
#include <cstring>
#include <string>
#include <unordered_set>
#include <vector>

#include "device_util.hpp"
#include "plan.hpp"

namespace remp {

// ---------------------------------------------------------------------------
// device data structures
// ---------------------------------------------------------------------------

// One live block of one sequence: physical block id, position of its first
// token on the sequence-major token axis, number of live tokens in it, and
// the sequence it belongs to.
struct BlockDesc {
    int32_t block;
    int32_t tok;
    int32_t n;
    int32_t seq;
};

constexpr bool kMergeRows = true;    // unpack whole destination rows when several sources fill them
// ... but only when every source's share of a row is at least this long: with
// short shares (GQA head rows of 256 B) alternating between staging streams
// within a row costs more read locality than whole-row writes gain (measured
// on MI355X: 70B GQA unpack 5.17 vs 5.32 TB/s; 7B MHA, 2 KiB shares, +1.3%).
constexpr uint32_t kMergeMinSegBytes = 1024;
// Slices per copy launch.  Launches of a few slices beat one launch of all of them (A/B on MI355X, 70B
// GQA share: 96 per launch 5.71, 40: 5.73, 10: 5.79-5.83, 5: 5.80, 2: 5.76, 1: 5.66 TB/s), and the kernel
// arguments stay small.
constexpr int kMaxItems = 8;
constexpr int kMaxUnitsPerWg = 128;   // (block, K or V) units per workgroup
// Copy launch policies (measured on MI355X).  Small (block, K/V) units, as
// with GQA head rows of 256 B, run fastest as many small workgroups, each
// moving one unit; large units (MHA rows of several KiB) prefer wider
// workgroups that move about 64 KiB.
constexpr int64_t kSmallUnitBytes = 16 * 1024;   // units up to this size use the small policy
constexpr int kSmallThreads = 128, kSmallUnroll = 4;
constexpr int kPackSmallThreads = 64, kPackSmallUnroll = 4;   // pack of small units: one wave per unit
// XCD-contiguous cell order, per launch kind (A/B on MI355X, one process: with it, 7B MHA pack
// +5%; 70B GQA small-unit pack -1.5% and unpack of block-sorted descriptors -1.6%)
constexpr bool kPackSmallXcd = false;
constexpr bool kUnpackSmallXcd = false;
constexpr bool kPackLargeXcd = true;
constexpr bool kUnpackLargeXcd = true;
constexpr int64_t kSmallWgBytes = 4 * 1024;
constexpr int64_t kLocalSmallWgBytes = 8 * 1024;   // the local copy's per-unit prologue wants 2 units (70B GQA: +14%)
constexpr int kLargeThreads = 256, kLargeUnroll = 8;
constexpr int64_t kLargeWgBytes = 64 * 1024;
constexpr int kScanThreads = 1024;

struct CopyItem {
    uint64_t paged_k;     // K storage of the layer, offset to the slice's first head
    uint64_t paged_v;
    uint64_t stage;       // first byte of the slice in its staging buffer (K part)
    uint32_t row_bytes;   // head_count * head_dim * elem_bytes
    uint32_t vpr_magic;   // fast division by vectors per row
    uint32_t unit_magic;  // fast division by vectors per (block, kv) unit
    uint16_t vpr_shift;
    uint16_t unit_shift;
};

struct CopyArgs {
    const BlockDesc* desc;
    int64_t block_stride;     // bytes per block on the paged side
    int64_t total_tokens;     // T: a slice's V part starts T * row_bytes after its K part
    int32_t n_desc;
    int32_t units_per_wg;
    int32_t row_stride;       // bytes per token row on the paged side (all local heads)
    int32_t block_size;       // paged-side block size
    CopyItem items[kMaxItems];
};
static_assert(sizeof(CopyArgs) < 4096, "copy kernel arguments must stay below 4 KiB");

// ---------------------------------------------------------------------------
// expansion: block tables -> one descriptor per live block
// ---------------------------------------------------------------------------

// Bucket of a physical block for the descriptor sort of the new tables (see
// below): nb buckets spread evenly over [0, num_blocks).
constexpr int kDescsPerBucket = 4;   // buckets = ceil(live blocks / 4): order kept at ~4-block granularity

__device__ __forceinline__ uint32_t block_bucket(int32_t block, int64_t num_blocks, uint32_t nb) {
    const int64_t b = static_cast<int64_t>(block > 0 ? block : 0) * nb / num_blocks;
    return static_cast<uint32_t>(b < nb ? b : nb - 1);
}

// Exclusive prefix sums of tokens and of blocks per sequence (one workgroup,
// wave64 shuffle scans combined through LDS, carried across chunks of 1024).
__global__ __launch_bounds__(kScanThreads) void expand_scan(const int32_t* __restrict__ lens, int32_t S,
                                                           int32_t bs, int32_t reset_flag, int32_t* __restrict__ flag,
                                                           int32_t* __restrict__ tok_off,
                                                           int32_t* __restrict__ blk_off,
                                                           int32_t* __restrict__ bucket, uint32_t nb) {
    __shared__ int64_t wave_tok[kScanThreads / 64];
    __shared__ int64_t wave_blk[kScanThreads / 64];
    __shared__ int64_t carry[2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) {
        carry[0] = 0;
        carry[1] = 0;
        if (reset_flag) *flag = 0;
    }
    if (bucket)   // counters of the descriptor sort, filled by expand_emit
        for (uint32_t i = tid; i < nb; i += kScanThreads) bucket[i] = 0;
    __syncthreads();
    bool bad = false;
    for (int32_t base = 0; base < S; base += kScanThreads) {
        const int32_t s = base + tid;
        int64_t n = s < S ? lens[s] : 0;
        if (n < 0) {
            n = 0;
            bad = true;
        }
        const int64_t nb = (n + bs - 1) / bs;
        int64_t it = n, ib = nb;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int64_t a = __shfl_up(it, d, 64);
            const int64_t b = __shfl_up(ib, d, 64);
            if (lane >= d) {
                it += a;
                ib += b;
            }
        }
        if (lane == 63) {
            wave_tok[wave] = it;
            wave_blk[wave] = ib;
        }
        __syncthreads();
        if (wave == 0) {
            const int nw = kScanThreads / 64;
            int64_t wt = lane < nw ? wave_tok[lane] : 0;
            int64_t wb = lane < nw ? wave_blk[lane] : 0;
#pragma unroll
            for (int d = 1; d < nw; d <<= 1) {
                const int64_t a = __shfl_up(wt, d, 64);
                const int64_t b = __shfl_up(wb, d, 64);
                if (lane >= d) {
                    wt += a;
                    wb += b;
                }
            }
            if (lane < nw) {   // exclusive totals of preceding waves
                wave_tok[lane] = wt;
                wave_blk[lane] = wb;
            }
        }
        __syncthreads();
        const int64_t pre_t = carry[0] + (wave ? wave_tok[wave - 1] : 0);
        const int64_t pre_b = carry[1] + (wave ? wave_blk[wave - 1] : 0);
        if (s < S) {
            const int64_t et = pre_t + it - n, eb = pre_b + ib - nb;
            if (et > INT32_MAX || eb > INT32_MAX) bad = true;
            tok_off[s] = static_cast<int32_t>(et < INT32_MAX ? et : INT32_MAX);
            blk_off[s] = static_cast<int32_t>(eb < INT32_MAX ? eb : INT32_MAX);
        }
        __syncthreads();
        if (tid == kScanThreads - 1) {
            carry[0] = pre_t + it;
            carry[1] = pre_b + ib;
        }
        __syncthreads();
    }
    if (tid == 0) {
        tok_off[S] = static_cast<int32_t>(carry[0] < INT32_MAX ? carry[0] : INT32_MAX);
        blk_off[S] = static_cast<int32_t>(carry[1] < INT32_MAX ? carry[1] : INT32_MAX);
    }
    if (bad) *flag = 1;
}

// One thread per live block: locate its sequence by binary search over the
// block offsets, then read its id from the table row.  Every index is bounded
// by the host-side sizes; an inconsistency yields an empty descriptor and sets
// the flag instead of an out-of-bounds access.
__global__ __launch_bounds__(256) void expand_emit(const int32_t* __restrict__ lens,
                                                   const int32_t* __restrict__ row_off,
                                                   const int32_t* __restrict__ ids, int32_t S, int32_t bs,
                                                   const int32_t* __restrict__ tok_off,
                                                   const int32_t* __restrict__ blk_off, int64_t nnz,
                                                   int64_t num_blocks, int64_t total_tokens, int64_t n_desc,
                                                   BlockDesc* __restrict__ desc, int32_t* __restrict__ flag,
                                                   int32_t* __restrict__ bucket, uint32_t nb) {
    const int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= n_desc) return;
    int32_t lo = 0, hi = S;   // last s in [0, S] with blk_off[s] <= b
    while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (blk_off[mid] <= b) lo = mid;
        else hi = mid - 1;
    }
    BlockDesc d{0, 0, 0, 0};
    bool ok = lo < S;
    if (ok) {
        const int32_t s = lo;
        const int64_t j = b - blk_off[s];
        const int64_t n = lens[s];
        const int64_t r = static_cast<int64_t>(row_off[s]) + j;
        ok = r >= 0 && r < nnz;
        if (ok) {
            const int64_t id = ids[r];
            const int64_t tok = static_cast<int64_t>(tok_off[s]) + j * bs;
            const int64_t rest = n - j * bs;
            const int64_t cnt = rest < bs ? rest : bs;
            ok = id >= 0 && id < num_blocks && cnt > 0 && tok >= 0 && tok + cnt <= total_tokens;
            if (ok) d = BlockDesc{static_cast<int32_t>(id), static_cast<int32_t>(tok), static_cast<int32_t>(cnt), s};
        }
    }
    if (!ok) *flag = 1;
    desc[b] = d;
    if (bucket) atomicAdd(&bucket[block_bucket(d.block, num_blocks > 0 ? num_blocks : 1, nb)], 1);
}

// ---------------------------------------------------------------------------
// ordering of the new descriptors by physical block
// ---------------------------------------------------------------------------

// The new tables come from a serving engine's free list, so consecutive live
// blocks sit at scattered physical addresses, and an unpack in descriptor
// order writes the pool in random 4-64 KiB pieces.  On MI355X random writes
// cost more than random reads (measured, 4 KiB pieces: 5.6 TB/s scattered
// writes against 6.1 TB/s scattered reads), so the new descriptors are
// bucket-sorted by block id first: the expansion clears and counts the
// buckets, then an exclusive scan and a scatter.  Order inside a bucket is
// whatever the atomics give; every order yields the same bytes.

// Exclusive scan of cnt[0, nb) in place (one workgroup, 4 consecutive counters
// per thread, carried over chunks of 4096).
constexpr int kSortScanPerThread = 4;

__global__ __launch_bounds__(kScanThreads) void sort_scan(int32_t* __restrict__ cnt, uint32_t nb) {
    __shared__ int32_t wave_sum[kScanThreads / 64];
    __shared__ int32_t carry;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) carry = 0;
    __syncthreads();
    for (uint32_t base = 0; base < nb; base += kScanThreads * kSortScanPerThread) {
        const uint32_t i0 = base + tid * kSortScanPerThread;
        int32_t c[kSortScanPerThread];
        int32_t v = 0;
#pragma unroll
        for (int k = 0; k < kSortScanPerThread; ++k) {
            c[k] = i0 + k < nb ? cnt[i0 + k] : 0;
            v += c[k];
        }
        int32_t x = v;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t a = __shfl_up(x, d, 64);
            if (lane >= d) x += a;
        }
        if (lane == 63) wave_sum[wave] = x;
        __syncthreads();
        if (wave == 0) {
            const int nw = kScanThreads / 64;
            int32_t w = lane < nw ? wave_sum[lane] : 0;
#pragma unroll
            for (int d = 1; d < nw; d <<= 1) {
                const int32_t a = __shfl_up(w, d, 64);
                if (lane >= d) w += a;
            }
            if (lane < nw) wave_sum[lane] = w;
        }
        __syncthreads();
        int32_t run = carry + (wave ? wave_sum[wave - 1] : 0) + x - v;   // exclusive prefix of counter i0
#pragma unroll
        for (int k = 0; k < kSortScanPerThread; ++k) {
            if (i0 + k < nb) cnt[i0 + k] = run;
            run += c[k];
        }
        const int32_t pre = carry + (wave ? wave_sum[wave - 1] : 0);
        __syncthreads();
        if (tid == kScanThreads - 1) carry = pre + x;
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void sort_scatter(const BlockDesc* __restrict__ desc, int32_t n, int64_t num_blocks,
                                                    uint32_t nb, int32_t* __restrict__ next,
                                                    BlockDesc* __restrict__ out) {
    const int32_t i = static_cast<int32_t>(blockIdx.x * 256 + threadIdx.x);
    if (i < n) {
        const BlockDesc d = desc[i];
        const int32_t pos = atomicAdd(&next[block_bucket(d.block, num_blocks, nb)], 1);
        if (pos >= 0 && pos < n) out[pos] = d;
    }
}

// ---------------------------------------------------------------------------
// pack / unpack copy
// ---------------------------------------------------------------------------


// Workgroup (x, y) of a grid -> the grid cell it works on.  With XCD, the
// cells are renumbered so that each of the 8 XCDs (the dispatcher deals
// workgroups to them round-robin in linear order) takes one contiguous range
// of cells: consecutive chunks of a slice then share an XCD's L2 and stream
// through neighbouring addresses.  A bijection of the grid onto itself.
template <bool XCD>
__device__ __forceinline__ void grid_cell(uint32_t* x, uint32_t* y) {
    *x = blockIdx.x;
    *y = blockIdx.y;
    if (XCD) {
        const uint32_t total = gridDim.x * gridDim.y;
        const uint32_t lin = blockIdx.y * gridDim.x + blockIdx.x;
        const uint32_t q = total / 8, r = total % 8, k = lin % 8;
        const uint32_t cell = k * q + min(k, r) + lin / 8;
        *x = cell % gridDim.x;
        *y = cell / gridDim.x;
    }
}

template <int VEC, bool PACK, int THREADS, int UNROLL, bool XCD>
__global__ __launch_bounds__(THREADS) void copy_slices(const CopyArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_paged[kMaxUnitsPerWg];
    __shared__ uint64_t s_stage[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];

    uint32_t cx, cy;
    grid_cell<XCD>(&cx, &cy);
    const CopyItem& it = args.items[cy];
    const int32_t u0 = static_cast<int32_t>(cx) * args.units_per_wg;
    const int32_t nu = min(args.units_per_wg, 2 * args.n_desc - u0);
    const int tid = threadIdx.x;
    const uint64_t kv_stride = static_cast<uint64_t>(args.total_tokens) * it.row_bytes;

    // unit u0 + u = (descriptor (u0 + u) / 2, kv = (u0 + u) % 2): base addresses of its two sides
    for (int u = tid; u < nu; u += THREADS) {
        const int32_t g = u0 + u;
        const BlockDesc d = args.desc[g >> 1];
        const int kv = g & 1;
        s_paged[u] = (kv ? it.paged_v : it.paged_k) + static_cast<uint64_t>(d.block) * args.block_stride;
        s_stage[u] = it.stage + kv * kv_stride + static_cast<uint64_t>(d.tok) * it.row_bytes;
        s_n[u] = d.n;
    }
    __syncthreads();

    const uint32_t vpr = it.row_bytes / VEC;
    const uint32_t unit = static_cast<uint32_t>(args.block_size) * vpr;
    const uint32_t total = static_cast<uint32_t>(nu) * unit;
    const uint32_t row_stride = static_cast<uint32_t>(args.row_stride);

    for (uint32_t base = tid; base < total; base += THREADS * UNROLL) {
        V r[UNROLL];
        uint64_t dst[UNROLL];
        bool ok[UNROLL];
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            const uint32_t idx = base + j * THREADS;
            ok[j] = false;
            dst[j] = 0;
            if (idx < total) {
                const uint32_t u = fast_div(idx, it.unit_magic, it.unit_shift);
                const uint32_t rem = idx - u * unit;
                const uint32_t row = fast_div(rem, it.vpr_magic, it.vpr_shift);
                const uint32_t c = rem - row * vpr;
                if (static_cast<int32_t>(row) < s_n[u]) {
                    const uint64_t paged = s_paged[u] + static_cast<uint64_t>(row) * row_stride + c * VEC;
                    const uint64_t stage = s_stage[u] + static_cast<uint64_t>(rem) * VEC;
                    const uint64_t src = PACK ? paged : stage;
                    dst[j] = PACK ? stage : paged;
                    r[j] = __builtin_nontemporal_load(reinterpret_cast<const V*>(src));
                    ok[j] = true;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < UNROLL; ++j)
            if (ok[j]) __builtin_nontemporal_store(r[j], reinterpret_cast<V*>(dst[j]));
    }
}


// Local copy (a slice whose old and new owner is the same rank): a unit is
// (new block, K or V); the prologue resolves every row of the unit's live
// tokens to its old (block, slot) through the old descriptors, so the main
// loop is a row-gather with one LDS lookup per vector.
constexpr int kMaxLocalItems = 8;     // local slices per launch (few per launch measured faster, as for kMaxItems)
constexpr int kMaxLocalRows = 1024;   // (unit, row) source addresses per workgroup

struct LocalItem {
    uint64_t src_k, src_v;   // old storage of the layer, offset to the slice's first head
    uint64_t dst_k, dst_v;   // new storage of the layer, offset to the slice's first head
    uint32_t row_bytes;
    uint32_t vpr_magic;
    uint32_t unit_magic;
    uint16_t vpr_shift;
    uint16_t unit_shift;
};

struct LocalArgs {
    const BlockDesc* new_desc;
    const BlockDesc* old_desc;
    const int32_t* tok_off;       // first token of each sequence on the token axis
    const int32_t* old_blk_off;   // first old descriptor of each sequence
    int32_t* flag;
    int64_t old_block_stride, new_block_stride;
    int32_t n_new_desc, n_old_desc;
    int32_t units_per_wg;
    int32_t old_row_stride, new_row_stride;
    int32_t old_block_size, new_block_size;
    LocalItem items[kMaxLocalItems];
};
static_assert(sizeof(LocalArgs) < 4096, "local copy kernel arguments must stay below 4 KiB");

template <int VEC, int THREADS, int UNROLL>
__global__ __launch_bounds__(THREADS) void copy_local(const LocalArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_dst[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ uint64_t s_src[kMaxLocalRows];

    const LocalItem& it = args.items[blockIdx.y];
    const int32_t u0 = static_cast<int32_t>(blockIdx.x) * args.units_per_wg;
    const int32_t nu = min(args.units_per_wg, 2 * args.n_new_desc - u0);
    const int tid = threadIdx.x;
    const int32_t bn = args.new_block_size, bo = args.old_block_size;

    for (int u = tid; u < nu; u += THREADS) {
        const int32_t g = u0 + u;
        const BlockDesc d = args.new_desc[g >> 1];
        s_dst[u] = ((g & 1) ? it.dst_v : it.dst_k) + static_cast<uint64_t>(d.block) * args.new_block_stride;
        s_n[u] = d.n;
    }
    for (int i = tid; i < nu * bn; i += THREADS) {
        const int32_t u = i / bn, r = i - u * bn;
        const int32_t g = u0 + u;
        const BlockDesc d = args.new_desc[g >> 1];
        uint64_t a = 0;
        if (r < d.n) {
            const int32_t t = d.tok - args.tok_off[d.seq] + r;          // token within its sequence
            const int32_t ob = args.old_blk_off[d.seq] + t / bo;
            const int32_t slot = t - (t / bo) * bo;
            bool ok = ob >= 0 && ob < args.n_old_desc;
            BlockDesc od{0, 0, 0, 0};
            if (ok) {
                od = args.old_desc[ob];
                ok = od.seq == d.seq && slot < od.n;
            }
            if (ok)
                a = ((g & 1) ? it.src_v : it.src_k) + static_cast<uint64_t>(od.block) * args.old_block_stride +
                    static_cast<uint64_t>(slot) * args.old_row_stride;
            else
                *args.flag = 1;
        }
        s_src[i] = a;
    }
    __syncthreads();

    const uint32_t vpr = it.row_bytes / VEC;
    const uint32_t unit = static_cast<uint32_t>(bn) * vpr;
    const uint32_t total = static_cast<uint32_t>(nu) * unit;
    const uint32_t new_row_stride = static_cast<uint32_t>(args.new_row_stride);
    for (uint32_t base = tid; base < total; base += THREADS * UNROLL) {
        V r[UNROLL];
        uint64_t dst[UNROLL];
        bool ok[UNROLL];
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            const uint32_t idx = base + j * THREADS;
            ok[j] = false;
            dst[j] = 0;
            if (idx < total) {
                const uint32_t u = fast_div(idx, it.unit_magic, it.unit_shift);
                const uint32_t rem = idx - u * unit;
                const uint32_t row = fast_div(rem, it.vpr_magic, it.vpr_shift);
                const uint32_t c = rem - row * vpr;
                const uint64_t src_row = s_src[u * bn + row];
                if (static_cast<int32_t>(row) < s_n[u] && src_row != 0) {
                    dst[j] = s_dst[u] + static_cast<uint64_t>(row) * new_row_stride + c * VEC;
                    r[j] = __builtin_nontemporal_load(reinterpret_cast<const V*>(src_row + c * VEC));
                    ok[j] = true;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < UNROLL; ++j)
            if (ok[j]) __builtin_nontemporal_store(r[j], reinterpret_cast<V*>(dst[j]));
    }
}


// ---------------------------------------------------------------------------
// head-tile copy through LDS, for pools whose token rows are not contiguous
// ---------------------------------------------------------------------------
//
// Layouts other than NHD keep each (block, head) as one contiguous tile of
// block_size * head_dim elements: HND stores it token-major ([slot][dim]);
// the ROCm paged-attention cache stores K as [dim / x][slot][x] (x = the
// elements in 16 bytes) and V as [dim][slot].  The staging side is always
// token-major.  A workgroup stages a few tiles in LDS in token-major order
// (rows padded by 16 bytes against bank conflicts), so both HBM sides are
// read and written as 16-byte vectors in their own contiguous order.

enum : int32_t { kLayoutNHD = 0, kLayoutHND = 1, kLayoutRocmSplit = 2 };
constexpr int kTileThreads = 256;
constexpr int kTileLdsBytes = 32 * 1024;   // dynamic LDS per workgroup, at most
constexpr int64_t kTileWgBytes = 16 * 1024; // payload bytes a tile workgroup aims to move

struct TileArgs {
    const BlockDesc* desc;
    int64_t block_stride;      // paged bytes per block
    int64_t total_tokens;
    int32_t n_desc;
    int32_t tiles_per_wg;
    int32_t block_size;
    int32_t head_bytes;        // head_dim * elem_bytes
    int32_t elem_bytes;
    int32_t layout;
    int32_t lds_row;           // head_bytes + 16
    uint32_t vpt_magic, vpt_shift;   // division by vectors per tile
    uint32_t vph_magic, vph_shift;   // division by vectors per head row
    uint32_t bs_magic, bs_shift;     // division by block_size
    CopyItem items[kMaxItems];       // paged_k/v: the slice's first head tile of the layer's block 0
};
static_assert(sizeof(TileArgs) < 4096, "tile kernel arguments must stay below 4 KiB");


// Move the elements of one 16-byte vector (consecutive slots of one dim) to or
// from LDS rows `lrow` bytes apart.
template <typename E>
__device__ __forceinline__ void scatter_t(const unsigned int __attribute__((ext_vector_type(4))) & val,
                                          unsigned char* p, uint32_t lrow) {
    const E* e = reinterpret_cast<const E*>(&val);
#pragma unroll
    for (int k = 0; k < 16 / static_cast<int>(sizeof(E)); ++k) *reinterpret_cast<E*>(p + k * lrow) = e[k];
}

template <typename E>
__device__ __forceinline__ unsigned int __attribute__((ext_vector_type(4))) gather_t(const unsigned char* p,
                                                                                      uint32_t lrow) {
    unsigned int __attribute__((ext_vector_type(4))) val;
    E* e = reinterpret_cast<E*>(&val);
#pragma unroll
    for (int k = 0; k < 16 / static_cast<int>(sizeof(E)); ++k) e[k] = *reinterpret_cast<const E*>(p + k * lrow);
    return val;
}

__device__ __forceinline__ void scatter_dim(const unsigned int __attribute__((ext_vector_type(4))) & val,
                                            unsigned char* p, uint32_t lrow, int32_t eb) {
    if (eb == 2) scatter_t<unsigned short>(val, p, lrow);
    else if (eb == 4) scatter_t<unsigned int>(val, p, lrow);
    else scatter_t<unsigned char>(val, p, lrow);
}

__device__ __forceinline__ unsigned int __attribute__((ext_vector_type(4))) gather_dim(const unsigned char* p,
                                                                                        uint32_t lrow, int32_t eb) {
    if (eb == 2) return gather_t<unsigned short>(p, lrow);
    if (eb == 4) return gather_t<unsigned int>(p, lrow);
    return gather_t<unsigned char>(p, lrow);
}

// Store the first `nbytes` bytes of a vector (whole elements of eb bytes).
__device__ __forceinline__ void store_prefix(const unsigned int __attribute__((ext_vector_type(4))) & val,
                                             void* dst, int32_t nbytes, int32_t eb) {
    const unsigned char* b = reinterpret_cast<const unsigned char*>(&val);
    unsigned char* o = reinterpret_cast<unsigned char*>(dst);
    if (eb == 4) {
        for (int q = 0; q < nbytes; q += 4)
            *reinterpret_cast<unsigned int*>(o + q) = *reinterpret_cast<const unsigned int*>(b + q);
    } else if (eb == 2) {
        for (int q = 0; q < nbytes; q += 2)
            *reinterpret_cast<unsigned short*>(o + q) = *reinterpret_cast<const unsigned short*>(b + q);
    } else {
        for (int q = 0; q < nbytes; ++q) o[q] = b[q];
    }
}

template <bool PACK>
__global__ __launch_bounds__(kTileThreads) void copy_tiles(const TileArgs args) {
    typedef unsigned int V4 __attribute__((ext_vector_type(4)));
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    __shared__ uint64_t s_paged[kMaxUnitsPerWg];
    __shared__ uint64_t s_stage[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ int32_t s_kv[kMaxUnitsPerWg];

    const CopyItem& it = args.items[blockIdx.y];
    const int32_t hc = static_cast<int32_t>(it.row_bytes) / args.head_bytes;   // heads in the slice
    const int64_t ntiles = static_cast<int64_t>(args.n_desc) * 2 * hc;
    const int64_t g0 = static_cast<int64_t>(blockIdx.x) * args.tiles_per_wg;
    if (g0 >= ntiles) return;
    const int32_t nt = static_cast<int32_t>(min(static_cast<int64_t>(args.tiles_per_wg), ntiles - g0));
    const int tid = threadIdx.x;
    const int32_t bs = args.block_size, hb = args.head_bytes;
    const uint64_t tile_bytes = static_cast<uint64_t>(bs) * hb;
    const uint64_t kv_stride = static_cast<uint64_t>(args.total_tokens) * it.row_bytes;

    for (int i = tid; i < nt; i += kTileThreads) {
        const int64_t g = g0 + i;
        const int64_t d = g / (2 * hc);
        const int32_t r = static_cast<int32_t>(g - d * 2 * hc);
        const int32_t kv = r / hc, j = r - (r / hc) * hc;
        const BlockDesc bd = args.desc[d];
        s_paged[i] = (kv ? it.paged_v : it.paged_k) + static_cast<uint64_t>(bd.block) * args.block_stride +
                     static_cast<uint64_t>(j) * tile_bytes;
        s_stage[i] = it.stage + kv * kv_stride + static_cast<uint64_t>(bd.tok) * it.row_bytes +
                     static_cast<uint64_t>(j) * hb;
        s_n[i] = bd.n;
        s_kv[i] = kv;
    }
    __syncthreads();

    const uint32_t vpt = static_cast<uint32_t>(tile_bytes / 16);     // 16-byte vectors per tile
    const uint32_t vph = static_cast<uint32_t>(hb / 16);             // 16-byte vectors per head row
    const uint32_t total = static_cast<uint32_t>(nt) * vpt;
    const uint32_t lrow = static_cast<uint32_t>(args.lds_row);
    const int32_t m = 16 / args.elem_bytes;                          // elements per vector
    const uint32_t tile_lds = static_cast<uint32_t>(bs) * lrow;

    // phase 1: fill LDS (token-major)
    for (uint32_t x = tid; x < total; x += kTileThreads) {
        const uint32_t i = fast_div(x, args.vpt_magic, args.vpt_shift);
        const uint32_t v = x - i * vpt;
        unsigned char* tl = lds + i * tile_lds;
        if (PACK) {
            const V4* src = reinterpret_cast<const V4*>(s_paged[i] + uint64_t(v) * 16);
            if (args.layout == kLayoutHND) {
                const uint32_t srow = fast_div(v, args.vph_magic, args.vph_shift);
                if (static_cast<int32_t>(srow) < s_n[i])
                    *reinterpret_cast<V4*>(tl + srow * lrow + (v - srow * vph) * 16) = __builtin_nontemporal_load(src);
            } else if (s_kv[i] == 0) {                                    // [dim / x][slot][x]
                const uint32_t c = fast_div(v, args.bs_magic, args.bs_shift);
                const uint32_t srow = v - c * bs;
                if (static_cast<int32_t>(srow) < s_n[i])
                    *reinterpret_cast<V4*>(tl + srow * lrow + c * 16) = __builtin_nontemporal_load(src);
            } else {                                                      // [dim][slot]
                const uint32_t e0 = v * m;
                const uint32_t dim = fast_div(e0, args.bs_magic, args.bs_shift);
                const uint32_t s0 = e0 - dim * bs;
                if (static_cast<int32_t>(s0) < s_n[i])
                    scatter_dim(__builtin_nontemporal_load(src), tl + s0 * lrow + dim * args.elem_bytes, lrow,
                                args.elem_bytes);
            }
        } else {
            const uint32_t srow = fast_div(v, args.vph_magic, args.vph_shift);
            const uint32_t cb = v - srow * vph;
            if (static_cast<int32_t>(srow) < s_n[i]) {
                const V4 val = __builtin_nontemporal_load(
                    reinterpret_cast<const V4*>(s_stage[i] + uint64_t(srow) * it.row_bytes + cb * 16));
                *reinterpret_cast<V4*>(tl + srow * lrow + cb * 16) = val;
            }
        }
    }
    __syncthreads();

    // phase 2: drain LDS
    for (uint32_t x = tid; x < total; x += kTileThreads) {
        const uint32_t i = fast_div(x, args.vpt_magic, args.vpt_shift);
        const uint32_t v = x - i * vpt;
        const unsigned char* tl = lds + i * tile_lds;
        if (PACK) {
            const uint32_t srow = fast_div(v, args.vph_magic, args.vph_shift);
            const uint32_t cb = v - srow * vph;
            if (static_cast<int32_t>(srow) < s_n[i])
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + srow * lrow + cb * 16),
                                            reinterpret_cast<V4*>(s_stage[i] + uint64_t(srow) * it.row_bytes + cb * 16));
        } else {
            V4* dst = reinterpret_cast<V4*>(s_paged[i] + uint64_t(v) * 16);
            if (args.layout == kLayoutHND) {
                const uint32_t srow = fast_div(v, args.vph_magic, args.vph_shift);
                if (static_cast<int32_t>(srow) < s_n[i])
                    __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + srow * lrow + (v - srow * vph) * 16), dst);
            } else if (s_kv[i] == 0) {
                const uint32_t c = fast_div(v, args.bs_magic, args.bs_shift);
                const uint32_t srow = v - c * bs;
                if (static_cast<int32_t>(srow) < s_n[i])
                    __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + srow * lrow + c * 16), dst);
            } else {
                const uint32_t e0 = v * m;
                const uint32_t dim = fast_div(e0, args.bs_magic, args.bs_shift);
                const uint32_t s0 = e0 - dim * bs;
                const int32_t live = min(m, s_n[i] - static_cast<int32_t>(s0));
                if (live <= 0) continue;
                const V4 val = gather_dim(tl + s0 * lrow + dim * args.elem_bytes, lrow, args.elem_bytes);
                if (live == m) {
                    __builtin_nontemporal_store(val, dst);
                } else {                                                  // only the live slots
                    store_prefix(val, dst, live * args.elem_bytes, args.elem_bytes);
                }
            }
        }
    }
}


// ---------------------------------------------------------------------------
// local copy between pools of any layouts, one head tile at a time through LDS
// ---------------------------------------------------------------------------
//
// A unit is one (new block, K or V, head of the slice) tile.  The prologue
// resolves each of its rows to the old (block, slot) through the old
// descriptors; phase 1 reads every live row's head vectors from the old pool
// in its layout into LDS (token-major); phase 2 writes the tile into the new
// pool in its layout, live slots only.  NHD rows on either side are read or
// written as 16-byte vectors of the row; the ROCm V layout, where a token's
// elements of one head lie block_size elements apart, is read element-wise.

constexpr int kMaxLocalTileItems = 8;

struct LocalTileItem {
    uint64_t src_k, src_v;   // old storage of the layer at the slice's first head (block 0)
    uint64_t dst_k, dst_v;   // new storage of the layer at the slice's first head (block 0)
    int32_t heads;           // heads in the slice
    int32_t pad;
};

struct LocalTileArgs {
    const BlockDesc* new_desc;
    const BlockDesc* old_desc;
    const int32_t* tok_off;       // first token of each sequence on the token axis
    const int32_t* old_blk_off;   // first old descriptor of each sequence
    int32_t* flag;
    int64_t old_block_stride, new_block_stride;   // bytes per block (all local heads)
    int32_t n_new_desc, n_old_desc;
    int32_t tiles_per_wg;
    int32_t old_block_size, new_block_size;
    int32_t head_bytes, elem_bytes;
    int32_t old_layout, new_layout;
    int32_t old_row_stride, new_row_stride;       // NHD: bytes per token row of all local heads
    int32_t old_head_step, new_head_step;         // bytes from one head's data to the next at block 0
    int32_t lds_row;                              // head_bytes + 16
    uint32_t vph_magic, vph_shift;                // division by vectors per head row
    uint32_t rows_magic, rows_shift;              // division by new_block_size * vectors per head row
    uint32_t bn_magic, bn_shift;                  // division by the new block size
    LocalTileItem items[kMaxLocalTileItems];
};
static_assert(sizeof(LocalTileArgs) < 4096, "local tile kernel arguments must stay below 4 KiB");

__global__ __launch_bounds__(kTileThreads) void copy_local_tiles(const LocalTileArgs a) {
    typedef unsigned int V4 __attribute__((ext_vector_type(4)));
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    __shared__ uint64_t s_dst[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ int32_t s_kv[kMaxUnitsPerWg];
    __shared__ uint64_t s_src[kMaxLocalRows];    // old tile (block, head) base of each (unit, row), 0: none
    __shared__ int32_t s_slot[kMaxLocalRows];

    const LocalTileItem& it = a.items[blockIdx.y];
    const int32_t hc = it.heads;
    const int64_t ntiles = static_cast<int64_t>(a.n_new_desc) * 2 * hc;
    const int64_t g0 = static_cast<int64_t>(blockIdx.x) * a.tiles_per_wg;
    if (g0 >= ntiles) return;
    const int32_t nt = static_cast<int32_t>(min(static_cast<int64_t>(a.tiles_per_wg), ntiles - g0));
    const int tid = threadIdx.x;
    const int32_t bn = a.new_block_size, bo = a.old_block_size, hb = a.head_bytes, eb = a.elem_bytes;

    for (int i = tid; i < nt; i += kTileThreads) {
        const int64_t g = g0 + i;
        const int64_t d = g / (2 * hc);
        const int32_t r = static_cast<int32_t>(g - d * 2 * hc);
        const int32_t kv = r / hc, j = r - (r / hc) * hc;
        const BlockDesc nd = a.new_desc[d];
        s_dst[i] = (kv ? it.dst_v : it.dst_k) + static_cast<uint64_t>(nd.block) * a.new_block_stride +
                   static_cast<uint64_t>(j) * a.new_head_step;
        s_n[i] = nd.n;
        s_kv[i] = kv;
    }
    for (int x = tid; x < nt * bn; x += kTileThreads) {
        const int32_t i = x / bn, r = x - (x / bn) * bn;
        const int64_t g = g0 + i;
        const int64_t d = g / (2 * hc);
        const int32_t rr = static_cast<int32_t>(g - d * 2 * hc);
        const int32_t kv = rr / hc, j = rr - (rr / hc) * hc;
        const BlockDesc nd = a.new_desc[d];
        uint64_t base = 0;
        int32_t slot = 0;
        if (r < nd.n) {
            const int32_t t = nd.tok - a.tok_off[nd.seq] + r;            // token within its sequence
            const int32_t ob = a.old_blk_off[nd.seq] + t / bo;
            slot = t - (t / bo) * bo;
            bool ok = ob >= 0 && ob < a.n_old_desc;
            BlockDesc od{0, 0, 0, 0};
            if (ok) {
                od = a.old_desc[ob];
                ok = od.seq == nd.seq && slot < od.n;
            }
            if (ok)
                base = (kv ? it.src_v : it.src_k) + static_cast<uint64_t>(od.block) * a.old_block_stride +
                       static_cast<uint64_t>(j) * a.old_head_step;
            else
                *a.flag = 1;
        }
        s_src[x] = base;
        s_slot[x] = slot;
    }
    __syncthreads();

    const uint32_t vph = static_cast<uint32_t>(hb / 16);
    const uint32_t per_tile = static_cast<uint32_t>(bn) * vph;
    const uint32_t total = static_cast<uint32_t>(nt) * per_tile;
    const uint32_t lrow = static_cast<uint32_t>(a.lds_row);
    const uint32_t tile_lds = static_cast<uint32_t>(bn) * lrow;
    const int32_t m = 16 / eb;                                      // elements per vector

    if (a.old_layout == a.new_layout && bo == bn) {
        // Same tile layout and block size: a new block holds the same tokens at the same slots as one
        // old block (blocks start at sequence starts), so each tile is copied vector for vector in
        // its own order, live slots only, without LDS.
        for (uint32_t x = tid; x < total; x += kTileThreads) {
            const uint32_t i = fast_div(x, a.rows_magic, a.rows_shift);
            const uint32_t v = x - i * per_tile;
            const int32_t n = s_n[i];
            const uint64_t src0 = s_src[i * bn];
            if (src0 == 0) continue;
            const V4* src = reinterpret_cast<const V4*>(src0 + uint64_t(v) * 16);
            V4* dst = reinterpret_cast<V4*>(s_dst[i] + uint64_t(v) * 16);
            if (a.new_layout == kLayoutHND || s_kv[i] == 0) {
                uint32_t r;
                if (a.new_layout == kLayoutHND) {
                    r = fast_div(v, a.vph_magic, a.vph_shift);
                } else {                                                 // [dim / x][slot][x]
                    const uint32_t c = fast_div(v, a.bn_magic, a.bn_shift);
                    r = v - c * bn;
                }
                if (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0)
                    __builtin_nontemporal_store(__builtin_nontemporal_load(src), dst);
            } else {                                                     // [dim][slot]
                const uint32_t e0 = v * m;
                const uint32_t dim = fast_div(e0, a.bn_magic, a.bn_shift);
                const uint32_t s0 = e0 - dim * bn;
                int32_t live = min(m, n - static_cast<int32_t>(s0));
                for (int k = 0; k < live; ++k)
                    if (s_src[i * bn + s0 + k] == 0) live = k;
                if (live <= 0) continue;
                const V4 val = __builtin_nontemporal_load(src);
                if (live == m) __builtin_nontemporal_store(val, dst);
                else store_prefix(val, dst, live * eb, eb);
            }
        }
        return;
    }

    // phase 1: live rows of every tile from the old pool into LDS, token-major
    for (uint32_t x = tid; x < total; x += kTileThreads) {
        const uint32_t i = fast_div(x, a.rows_magic, a.rows_shift);
        const uint32_t rem = x - i * per_tile;
        const uint32_t r = fast_div(rem, a.vph_magic, a.vph_shift);
        const uint32_t c = rem - r * vph;
        const uint64_t base = s_src[i * bn + r];
        if (static_cast<int32_t>(r) >= s_n[i] || base == 0) continue;
        const uint32_t slot = static_cast<uint32_t>(s_slot[i * bn + r]);
        V4 val;
        if (a.old_layout == kLayoutNHD) {
            val = __builtin_nontemporal_load(reinterpret_cast<const V4*>(base + uint64_t(slot) * a.old_row_stride + c * 16));
        } else if (a.old_layout == kLayoutHND) {
            val = __builtin_nontemporal_load(reinterpret_cast<const V4*>(base + uint64_t(slot) * hb + c * 16));
        } else if (s_kv[i] == 0) {                                       // [dim / x][slot][x]
            val = __builtin_nontemporal_load(reinterpret_cast<const V4*>(base + uint64_t(c) * bo * 16 + slot * 16));
        } else {                                                         // [dim][slot]: element-wise
            unsigned char* vb = reinterpret_cast<unsigned char*>(&val);
            const unsigned char* src = reinterpret_cast<const unsigned char*>(base) + uint64_t(c) * m * bo * eb +
                                       uint64_t(slot) * eb;
            for (int k = 0; k < m; ++k) {
                const unsigned char* e = src + uint64_t(k) * bo * eb;
                if (eb == 2) *reinterpret_cast<unsigned short*>(vb + 2 * k) = *reinterpret_cast<const unsigned short*>(e);
                else if (eb == 4) *reinterpret_cast<unsigned int*>(vb + 4 * k) = *reinterpret_cast<const unsigned int*>(e);
                else vb[k] = *e;
            }
        }
        *reinterpret_cast<V4*>(lds + i * tile_lds + r * lrow + c * 16) = val;
    }
    __syncthreads();

    // phase 2: every tile into the new pool in its layout, live slots only
    for (uint32_t x = tid; x < total; x += kTileThreads) {
        const uint32_t i = fast_div(x, a.rows_magic, a.rows_shift);
        const uint32_t v = x - i * per_tile;                            // vector of the tile in its own order
        const unsigned char* tl = lds + i * tile_lds;
        const int32_t n = s_n[i];
        if (a.new_layout == kLayoutNHD) {
            const uint32_t r = fast_div(v, a.vph_magic, a.vph_shift);
            const uint32_t c = v - r * vph;
            if (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0)
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + r * lrow + c * 16),
                                            reinterpret_cast<V4*>(s_dst[i] + uint64_t(r) * a.new_row_stride + c * 16));
            continue;
        }
        V4* dst = reinterpret_cast<V4*>(s_dst[i] + uint64_t(v) * 16);
        if (a.new_layout == kLayoutHND) {
            const uint32_t r = fast_div(v, a.vph_magic, a.vph_shift);
            if (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0)
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + r * lrow + (v - r * vph) * 16), dst);
        } else if (s_kv[i] == 0) {                                       // [dim / x][slot][x]
            const uint32_t c = fast_div(v, a.bn_magic, a.bn_shift);
            const uint32_t r = v - c * bn;
            if (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0)
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + r * lrow + c * 16), dst);
        } else {                                                         // [dim][slot]
            const uint32_t e0 = v * m;
            const uint32_t dim = fast_div(e0, a.bn_magic, a.bn_shift);
            const uint32_t s0 = e0 - dim * bn;
            int32_t live = min(m, n - static_cast<int32_t>(s0));
            for (int k = 0; k < live; ++k)                              // rows without a source stay untouched
                if (s_src[i * bn + s0 + k] == 0) live = k;
            if (live <= 0) continue;
            const V4 val = gather_dim(tl + s0 * lrow + dim * eb, lrow, eb);
            if (live == m) __builtin_nontemporal_store(val, dst);
            else store_prefix(val, dst, live * eb, eb);
        }
    }
}


// ---------------------------------------------------------------------------
// unpack with whole destination rows
// ---------------------------------------------------------------------------
//
// When a new rank receives a layer's heads from several sources, the plain
// unpack writes each source's head range as its own pass over the new blocks,
// so every block row is opened once per source.  This variant takes one
// (layer, new block, K/V) unit per workgroup and writes the unit's rows whole:
// each 16-byte vector of a row finds the source slice holding its head and
// reads it from that slice's staging.  All layers of a call share the split of
// the row into source slices.

constexpr int kMaxMergeSegs = 8;
constexpr int kMaxMergeGroups = 8;

struct MergeSeg {
    uint32_t row_bytes;   // head_count * head_bytes of the slice
    uint16_t head0;       // first local head
    uint16_t head_count;
};

struct MergeArgs {
    const BlockDesc* desc;
    int64_t block_stride;
    int64_t total_tokens;
    int32_t n_desc;
    int32_t units_per_wg;
    int32_t row_stride;       // full destination row
    int32_t block_size;
    int32_t nseg;
    int32_t head_bytes;
    uint32_t vpr_magic, vpr_shift;     // vectors per full row
    uint32_t unit_magic, unit_shift;   // vectors per (block, K/V) unit
    uint32_t vph_magic, vph_shift;     // vectors per head
    MergeSeg segs[kMaxMergeSegs];
    uint64_t paged_k[kMaxMergeGroups];
    uint64_t paged_v[kMaxMergeGroups];
    uint64_t stage[kMaxMergeGroups][kMaxMergeSegs / 2];   // filled for nseg <= kMaxMergeSegs / 2
};
static_assert(sizeof(MergeArgs) < 4096, "merged unpack kernel arguments must stay below 4 KiB");

template <int VEC, int THREADS, int UNROLL>
__global__ __launch_bounds__(THREADS) void unpack_rows(const MergeArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_paged[kMaxUnitsPerWg];
    __shared__ int32_t s_tok[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ int32_t s_kv[kMaxUnitsPerWg];

    const int32_t g = blockIdx.y;
    const int32_t u0 = static_cast<int32_t>(blockIdx.x) * args.units_per_wg;
    const int32_t nu = min(args.units_per_wg, 2 * args.n_desc - u0);
    const int tid = threadIdx.x;
    for (int u = tid; u < nu; u += THREADS) {
        const int32_t x = u0 + u;
        const BlockDesc d = args.desc[x >> 1];
        const int kv = x & 1;
        s_paged[u] = (kv ? args.paged_v[g] : args.paged_k[g]) + static_cast<uint64_t>(d.block) * args.block_stride;
        s_tok[u] = d.tok;
        s_n[u] = d.n;
        s_kv[u] = kv;
    }
    __syncthreads();

    const uint32_t vpr = static_cast<uint32_t>(args.row_stride) / VEC;
    const uint32_t vph = static_cast<uint32_t>(args.head_bytes) / VEC;
    const uint32_t unit = static_cast<uint32_t>(args.block_size) * vpr;
    const uint32_t total = static_cast<uint32_t>(nu) * unit;
    for (uint32_t base = tid; base < total; base += THREADS * UNROLL) {
        V r[UNROLL];
        uint64_t dst[UNROLL];
        bool ok[UNROLL];
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            const uint32_t idx = base + j * THREADS;
            ok[j] = false;
            dst[j] = 0;
            if (idx < total) {
                const uint32_t u = fast_div(idx, args.unit_magic, args.unit_shift);
                const uint32_t rem = idx - u * unit;
                const uint32_t row = fast_div(rem, args.vpr_magic, args.vpr_shift);
                const uint32_t c = rem - row * vpr;
                if (static_cast<int32_t>(row) < s_n[u]) {
                    const uint32_t h = fast_div(c, args.vph_magic, args.vph_shift);
                    int32_t sg = 0;
                    while (sg + 1 < args.nseg && h >= args.segs[sg + 1].head0) ++sg;
                    const MergeSeg seg = args.segs[sg];
                    const uint64_t src = args.stage[g][sg] +
                                         static_cast<uint64_t>(s_kv[u]) * args.total_tokens * seg.row_bytes +
                                         static_cast<uint64_t>(s_tok[u] + row) * seg.row_bytes +
                                         static_cast<uint64_t>(h - seg.head0) * args.head_bytes +
                                         (c - h * vph) * VEC;
                    dst[j] = s_paged[u] + static_cast<uint64_t>(row) * args.row_stride + c * VEC;
                    r[j] = __builtin_nontemporal_load(reinterpret_cast<const V*>(src));
                    ok[j] = true;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < UNROLL; ++j)
            if (ok[j]) __builtin_nontemporal_store(r[j], reinterpret_cast<V*>(dst[j]));
    }
}

// ---------------------------------------------------------------------------
// host launch code
// ---------------------------------------------------------------------------

static thread_local hipEvent_t g_trace_start = nullptr;
static thread_local hipEvent_t g_trace_stop = nullptr;

static int env_int(const char* name, int dflt) {
    const char* v = std::getenv(name);
    if (!v || !*v) return dflt;
    return std::atoi(v);
}

struct HostSlice {
    uint64_t paged_k, paged_v, stage;
    uint32_t row_bytes;
    int32_t layer = 0;        // global layer
    int32_t head_local = 0;   // first head of the slice within the paged rank's heads
    int32_t head_count = 0;
    uint64_t layer_k = 0, layer_v = 0;   // the layer's storage (no head offset)
};


static uint32_t sort_buckets(int64_t n_desc) {
    return static_cast<uint32_t>((std::max<int64_t>(n_desc, 1) + kDescsPerBucket - 1) / kDescsPerBucket);
}

// Enqueue expansion of `tables` into the workspace areas at scan_off / desc_off.
// With bucket_off >= 0 the expansion also clears and fills the bucket counters
// of the descriptor sort (new tables only).
static remp_status launch_expand(const remp_kv_plan_t& p, const remp_dev_tables& dt, int32_t bs, int64_t nnz,
                                 int64_t num_blocks, int64_t n_desc, char* ws, int64_t scan_off, int64_t desc_off,
                                 bool reset_flag, hipStream_t stream, int64_t bucket_off = -1) {
    if (n_desc >= (int64_t(1) << 30)) return fail(REMP_E_UNSUPPORTED, "more than 2^30 live blocks in one call");
    int32_t* flag = reinterpret_cast<int32_t*>(ws);
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
                           p.total_tokens, n_desc, desc, flag, bucket, nb);
        if (remp_status st = hip_check(hipGetLastError(), "expand_emit launch")) return st;
    }
    return REMP_OK;
}

// Finish the bucket sort of the n_desc new descriptors at desc_off (counted by
// the expansion into bucket_off) into sorted_off.
static remp_status launch_sort_new(int64_t n_desc, int64_t num_blocks, char* ws, int64_t desc_off,
                                   int64_t bucket_off, int64_t sorted_off, hipStream_t stream) {
    if (n_desc <= 0) return REMP_OK;
    const uint32_t nb = sort_buckets(n_desc);
    const uint32_t grid = static_cast<uint32_t>((n_desc + 255) / 256);
    const BlockDesc* desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    int32_t* cnt = reinterpret_cast<int32_t*>(ws + bucket_off);
    BlockDesc* out = reinterpret_cast<BlockDesc*>(ws + sorted_off);
    const int64_t nblk = num_blocks > 0 ? num_blocks : 1;
    hipLaunchKernelGGL(sort_scan, dim3(1), dim3(kScanThreads), 0, stream, cnt, nb);
    hipLaunchKernelGGL(sort_scatter, dim3(grid), dim3(256), 0, stream, desc, static_cast<int32_t>(n_desc), nblk, nb,
                       cnt, out);
    return hip_check(hipGetLastError(), "descriptor sort launch");
}

// Launch shapes measured on MI355X (70B GQA and 7B MHA shares): small-unit pack runs one wave per
// 4 KiB unit in plain grid order; everything else takes the XCD-contiguous cell order.
template <int VEC, bool PACK>
static void launch_copy_vec(const CopyArgs& a, dim3 grid, bool small, hipStream_t stream) {
    if (small && PACK)
        hipLaunchKernelGGL((copy_slices<VEC, true, kPackSmallThreads, kPackSmallUnroll, kPackSmallXcd>), grid,
                           dim3(kPackSmallThreads), 0, stream, a);
    else if (small)
        hipLaunchKernelGGL((copy_slices<VEC, false, kSmallThreads, kSmallUnroll, kUnpackSmallXcd>), grid,
                           dim3(kSmallThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((copy_slices<VEC, PACK, kLargeThreads, kLargeUnroll, PACK ? kPackLargeXcd : kUnpackLargeXcd>),
                           grid, dim3(kLargeThreads), 0, stream, a);
}

template <bool PACK>
static remp_status launch_copy(const remp_kv_plan_t& p, const std::vector<HostSlice>& slices, int64_t n_desc,
                               int32_t bs, int64_t block_stride, int32_t row_stride, const char* ws,
                               int64_t desc_off, hipStream_t stream) {
    if (slices.empty() || n_desc == 0) return REMP_OK;
    if (n_desc >= (int64_t(1) << 30)) return fail(REMP_E_UNSUPPORTED, "more than 2^30 live blocks in one call");
    // widest vector every address and stride is aligned to
    uint64_t bits = static_cast<uint64_t>(block_stride) | static_cast<uint64_t>(row_stride) | 16u;
    uint32_t max_row = 0;
    for (const HostSlice& s : slices) {
        bits |= s.paged_k | s.paged_v | s.stage | s.row_bytes |
                (static_cast<uint64_t>(p.total_tokens) * s.row_bytes);
        max_row = std::max(max_row, s.row_bytes);
    }
    const int vec = static_cast<int>(bits & (~bits + 1));   // lowest set bit, <= 16
    const int64_t per_unit = static_cast<int64_t>(bs) * max_row;
    const bool small = per_unit <= kSmallUnitBytes;
    const int64_t target = env_int("REMP_KV_WG_BYTES", static_cast<int>(small ? kSmallWgBytes : kLargeWgBytes));
    int32_t C = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(kMaxUnitsPerWg, target / per_unit)));
    // the flattened per-workgroup index must stay below 2^32
    while (C > 1 && static_cast<uint64_t>(C) * bs * (max_row / vec) >= (uint64_t(1) << 32)) C >>= 1;
    if (static_cast<uint64_t>(bs) * (max_row / vec) >= (uint64_t(1) << 32))
        return fail(REMP_E_UNSUPPORTED, "a block of one slice exceeds 2^32 vectors");

    CopyArgs a;
    std::memset(&a, 0, sizeof(a));
    a.desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    a.block_stride = block_stride;
    a.total_tokens = p.total_tokens;
    a.n_desc = static_cast<int32_t>(n_desc);
    a.units_per_wg = C;
    a.row_stride = row_stride;
    a.block_size = bs;
    const int64_t gx = (2 * n_desc + C - 1) / C;
    if (gx * kMaxItems >= (int64_t(1) << 32))
        return fail(REMP_E_UNSUPPORTED, "too many block descriptors for one launch");

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
            case 16: launch_copy_vec<16, PACK>(a, grid, small, stream); break;
            case 8: launch_copy_vec<8, PACK>(a, grid, small, stream); break;
            case 4: launch_copy_vec<4, PACK>(a, grid, small, stream); break;
            case 2: launch_copy_vec<2, PACK>(a, grid, small, stream); break;
            default: launch_copy_vec<1, PACK>(a, grid, small, stream); break;
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
                                hipStream_t stream) {
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
    if (gx > 0x7FFFFFFF) return fail(REMP_E_UNSUPPORTED, "too many tiles for one launch");

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


// Unpack with whole destination rows, when every layer of the call receives
// the same split of its rows into 2..kMaxMergeSegs/2 source slices covering
// all of the rank's heads.  Returns false (nothing enqueued) if not applicable.
template <int VEC>
static void launch_rows_vec(const MergeArgs& a, dim3 grid, bool small, hipStream_t stream) {
    if (small)
        hipLaunchKernelGGL((unpack_rows<VEC, kSmallThreads, kSmallUnroll>), grid, dim3(kSmallThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((unpack_rows<VEC, kLargeThreads, kLargeUnroll>), grid, dim3(kLargeThreads), 0, stream, a);
}

static bool merged_rows_apply(const std::vector<HostSlice>& slices, int32_t heads_per_rank,
                              std::vector<std::vector<const HostSlice*>>& groups) {
    std::vector<int32_t> layers;
    for (const HostSlice& s : slices)
        if (std::find(layers.begin(), layers.end(), s.layer) == layers.end()) layers.push_back(s.layer);
    groups.clear();
    for (int32_t l : layers) {
        std::vector<const HostSlice*> g;
        for (const HostSlice& s : slices)
            if (s.layer == l) g.push_back(&s);
        std::sort(g.begin(), g.end(), [](const HostSlice* a, const HostSlice* b) { return a->head_local < b->head_local; });
        if (g.size() < 2 || g.size() > kMaxMergeSegs / 2) return false;
        int32_t next = 0;                                 // slices tile the rank's heads exactly
        for (const HostSlice* s : g) {
            if (s->head_local != next || s->row_bytes < kMergeMinSegBytes) return false;
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

static remp_status launch_rows(const remp_kv_plan_t& p, const std::vector<std::vector<const HostSlice*>>& groups,
                               int64_t n_desc, int32_t bs, int64_t block_stride, int32_t row_stride, const char* ws,
                               int64_t desc_off, hipStream_t stream) {
    if (groups.empty() || n_desc == 0) return REMP_OK;
    const int64_t hb = static_cast<int64_t>(p.shape.head_dim) * p.shape.elem_bytes;
    uint64_t bits = static_cast<uint64_t>(block_stride) | static_cast<uint64_t>(row_stride) |
                    static_cast<uint64_t>(hb) | 16u;
    for (const auto& g : groups)
        for (const HostSlice* s : g)
            bits |= s->layer_k | s->layer_v | s->stage | s->row_bytes |
                    (static_cast<uint64_t>(p.total_tokens) * s->row_bytes);
    const int vec = static_cast<int>(bits & (~bits + 1));
    const int64_t per_unit = static_cast<int64_t>(bs) * row_stride;
    const bool small = per_unit <= kSmallUnitBytes;
    const int64_t target = env_int("REMP_KV_WG_BYTES", static_cast<int>(small ? kSmallWgBytes : kLargeWgBytes));
    int32_t C = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(kMaxUnitsPerWg, target / per_unit)));
    while (C > 1 && static_cast<uint64_t>(C) * bs * (row_stride / vec) >= (uint64_t(1) << 32)) C >>= 1;
    if (static_cast<uint64_t>(bs) * (row_stride / vec) >= (uint64_t(1) << 32))
        return fail(REMP_E_UNSUPPORTED, "a block of one row exceeds 2^32 vectors");
    MergeArgs a;
    std::memset(&a, 0, sizeof(a));
    a.desc = reinterpret_cast<const BlockDesc*>(ws + desc_off);
    a.block_stride = block_stride;
    a.total_tokens = p.total_tokens;
    a.n_desc = static_cast<int32_t>(n_desc);
    a.units_per_wg = C;
    a.row_stride = row_stride;
    a.block_size = bs;
    a.head_bytes = static_cast<int32_t>(hb);
    const auto& first = groups.front();
    a.nseg = static_cast<int32_t>(first.size());
    for (size_t i = 0; i < first.size(); ++i)
        a.segs[i] = MergeSeg{first[i]->row_bytes, static_cast<uint16_t>(first[i]->head_local),
                             static_cast<uint16_t>(first[i]->head_count)};
    const FastDiv fv = make_fastdiv(static_cast<uint32_t>(row_stride / vec));
    const FastDiv fu = make_fastdiv(static_cast<uint32_t>(bs) * static_cast<uint32_t>(row_stride / vec));
    const FastDiv fh = make_fastdiv(static_cast<uint32_t>(hb / vec));
    a.vpr_magic = fv.magic;
    a.vpr_shift = fv.shift;
    a.unit_magic = fu.magic;
    a.unit_shift = fu.shift;
    a.vph_magic = fh.magic;
    a.vph_shift = fh.shift;
    const int64_t gx = (2 * n_desc + C - 1) / C;
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
            case 16: launch_rows_vec<16>(a, grid, small, stream); break;
            case 8: launch_rows_vec<8>(a, grid, small, stream); break;
            case 4: launch_rows_vec<4>(a, grid, small, stream); break;
            case 2: launch_rows_vec<2>(a, grid, small, stream); break;
            default: launch_rows_vec<1>(a, grid, small, stream); break;
        }
        if (remp_status st = hip_check(hipGetLastError(), "unpack rows launch")) return st;
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
                                    const remp_kv_pool* dst, int64_t* nnz_out) {
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
    for (int32_t q = 0; q < t.num_seqs; ++q) {
        if (t.seq_lens[q] != plan->seq_lens[q])
            return fail(REMP_E_INVALID, "new tables give sequence " + std::to_string(q) + " length " +
                                            std::to_string(t.seq_lens[q]) + ", planned " +
                                            std::to_string(plan->seq_lens[q]));
        const int32_t a = t.row_offsets[q], b = t.row_offsets[q + 1];
        if (b < a) return fail(REMP_E_INVALID, "new row_offsets decrease at sequence " + std::to_string(q));
        const int64_t need = ceil_div(t.seq_lens[q], sh.new_block_size);
        if (b - a < need) return fail(REMP_E_INVALID, "new table row of sequence " + std::to_string(q) + " too short");
        for (int64_t j = 0; j < need; ++j) {
            const int32_t id = t.block_ids[a + j];
            if (id < 0 || id >= t.num_blocks)
                return fail(REMP_E_RANGE, "new block id " + std::to_string(id) + " outside [0, " +
                                              std::to_string(t.num_blocks) + ")");
            if (used[id]) return fail(REMP_E_INVALID, "new block id " + std::to_string(id) + " used twice");
            used[id] = 1;
        }
    }
    *nnz_out = nnz;
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
        hipLaunchKernelGGL((copy_local<VEC, kSmallThreads, kSmallUnroll>), grid, dim3(kSmallThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((copy_local<VEC, kLargeThreads, kLargeUnroll>), grid, dim3(kLargeThreads), 0, stream, a);
    return hip_check(hipGetLastError(), "copy_local launch");
}

// Local copy when either pool is not NHD: head tiles through LDS.  items carry
// the slice's first-head offsets in each pool's own layout.
static remp_status launch_local_tiles(const remp_kv_plan_t& p, const std::vector<HostLocal>& items,
                                      int32_t old_layout, int32_t new_layout, const char* ws, hipStream_t stream) {
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
    a.tok_off = reinterpret_cast<const int32_t*>(ws + L.scan_new);
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
        if (gx > 0x7FFFFFFF) return fail(REMP_E_UNSUPPORTED, "too many head tiles for one launch");
        // 32-bit vector indices per workgroup: T tiles of bn rows of hb / 16 vectors
        hipLaunchKernelGGL(copy_local_tiles, dim3(static_cast<uint32_t>(gx), static_cast<uint32_t>(cnt)),
                           dim3(kTileThreads), static_cast<size_t>(T * tile_lds), stream, a);
        if (remp_status st = hip_check(hipGetLastError(), "copy_local_tiles launch")) return st;
    }
    if (g_trace_stop) {
        if (remp_status st = hip_check(hipEventRecord(g_trace_stop, stream), "trace stop event")) return st;
    }
    return REMP_OK;
}

static remp_status launch_local(const remp_kv_plan_t& p, const std::vector<HostLocal>& items, const char* ws,
                                hipStream_t stream) {
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
    const int64_t target = env_int("REMP_KV_WG_BYTES", static_cast<int>(small ? kLocalSmallWgBytes : kLargeWgBytes));
    int32_t C = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(kMaxUnitsPerWg, target / per_unit)));
    C = std::min<int32_t>(C, std::max<int32_t>(1, kMaxLocalRows / bn));
    if (bn > kMaxLocalRows) return fail(REMP_E_UNSUPPORTED, "new block size above the local-copy row limit");
    if (static_cast<uint64_t>(C) * bn * (max_row / vec) >= (uint64_t(1) << 32))
        return fail(REMP_E_UNSUPPORTED, "a block of one slice exceeds 2^32 vectors");

    LocalArgs a;
    std::memset(&a, 0, sizeof(a));
    a.new_desc = reinterpret_cast<const BlockDesc*>(ws + L.sorted_new);
    a.old_desc = reinterpret_cast<const BlockDesc*>(ws + L.desc_old);
    a.tok_off = reinterpret_cast<const int32_t*>(ws + L.scan_new);
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
    const int64_t gx = (2 * n_desc + C - 1) / C;
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
    if (flags & ~static_cast<uint32_t>(REMP_KV_SKIP_LOCAL)) return fail(REMP_E_INVALID, "unknown flags");
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
    if (slices.empty() || plan->old_live_blocks == 0) return REMP_OK;
    const remp_kv_shape& sh = plan->shape;
    const int64_t row_stride = static_cast<int64_t>(plan->own_old.heads_per_rank()) * sh.head_dim * sh.elem_bytes;
    const WorkspaceLayout L = workspace_layout(*plan);
    char* ws = static_cast<char*>(workspace);
    if (remp_status st = launch_expand(*plan, *old_tables, sh.old_block_size, plan->old_nnz, plan->old_num_blocks,
                                       plan->old_live_blocks, ws, L.scan_old, L.desc_old, true, stream))
        return st;
    if (src->layout != kLayoutNHD)
        return launch_tiles<true>(*plan, slices, plan->old_live_blocks, sh.old_block_size,
                                  row_stride * sh.old_block_size, src->layout, ws, L.desc_old, stream);
    return launch_copy<true>(*plan, slices, plan->old_live_blocks, sh.old_block_size, row_stride * sh.old_block_size,
                             static_cast<int32_t>(row_stride), ws, L.desc_old, stream);
}

remp_status remp_kv_unpack(const remp_kv_plan_t* plan, int32_t new_rank, int32_t layer_begin, int32_t layer_end,
                           const remp_buffer* staging, const remp_kv_pool* dst, const remp_block_tables* new_tables,
                           const remp_dev_tables* new_dev_tables, void* workspace, int64_t workspace_bytes_,
                           uint32_t flags, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    if (flags & ~static_cast<uint32_t>(REMP_KV_SKIP_LOCAL)) return fail(REMP_E_INVALID, "unknown flags");
    if (new_rank < 0 || new_rank >= plan->own_new.world())
        return fail(REMP_E_RANGE, "new_rank " + std::to_string(new_rank) + " outside [0, " +
                                      std::to_string(plan->own_new.world()) + ")");
    if (remp_status st = check_window(plan, layer_begin, layer_end)) return st;
    if (remp_status st = check_pool(plan, dst, plan->own_new.layers_of_rank(new_rank), plan->shape.new_block_size,
                                    "destination"))
        return st;
    if (!staging) return fail(REMP_E_INVALID, "staging array is NULL");
    if (remp_status st = check_workspace(plan, workspace, workspace_bytes_)) return st;
    int64_t nnz = 0;
    if (remp_status st = check_new_tables(plan, new_tables, dst, &nnz)) return st;
    if (remp_status st = check_dev_tables(plan, new_dev_tables, nnz, "new")) return st;

    std::vector<HostSlice> slices;
    if (remp_status st = collect_slices(*plan, false, new_rank, layer_begin, layer_end, *dst, staging,
                                        (flags & REMP_KV_SKIP_LOCAL) != 0, slices))
        return st;
    if (slices.empty() || plan->new_live_blocks == 0) return REMP_OK;
    const remp_kv_shape& sh = plan->shape;
    const int64_t row_stride = static_cast<int64_t>(plan->own_new.heads_per_rank()) * sh.head_dim * sh.elem_bytes;
    const WorkspaceLayout L = workspace_layout(*plan);
    char* ws = static_cast<char*>(workspace);
    if (remp_status st = launch_expand(*plan, *new_dev_tables, sh.new_block_size, nnz, new_tables->num_blocks,
                                       plan->new_live_blocks, ws, L.scan_new, L.desc_new, true, stream, L.bucket_new))
        return st;
    if (remp_status st = launch_sort_new(plan->new_live_blocks, new_tables->num_blocks, ws, L.desc_new, L.bucket_new,
                                         L.sorted_new, stream))
        return st;
    if (dst->layout != kLayoutNHD)
        return launch_tiles<false>(*plan, slices, plan->new_live_blocks, sh.new_block_size,
                                   row_stride * sh.new_block_size, dst->layout, ws, L.sorted_new, stream);
    std::vector<std::vector<const HostSlice*>> groups;
    if (kMergeRows && merged_rows_apply(slices, plan->own_new.heads_per_rank(), groups))
        return launch_rows(*plan, groups, plan->new_live_blocks, sh.new_block_size, row_stride * sh.new_block_size,
                           static_cast<int32_t>(row_stride), ws, L.sorted_new, stream);
    return launch_copy<false>(*plan, slices, plan->new_live_blocks, sh.new_block_size, row_stride * sh.new_block_size,
                              static_cast<int32_t>(row_stride), ws, L.sorted_new, stream);
}

remp_status remp_kv_copy_local(const remp_kv_plan_t* plan, int32_t rank, int32_t layer_begin, int32_t layer_end,
                               const remp_kv_pool* src, const remp_dev_tables* old_tables, const remp_kv_pool* dst,
                               const remp_block_tables* new_tables, const remp_dev_tables* new_dev_tables,
                               void* workspace, int64_t workspace_bytes_, hipStream_t stream) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
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
    if (remp_status st = check_new_tables(plan, new_tables, dst, &nnz)) return st;
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
    if (items.empty() || plan->new_live_blocks == 0) return REMP_OK;
    const WorkspaceLayout L = workspace_layout(*plan);
    char* ws = static_cast<char*>(workspace);
    if (remp_status st = launch_expand(*plan, *old_tables, sh.old_block_size, plan->old_nnz, plan->old_num_blocks,
                                       plan->old_live_blocks, ws, L.scan_old, L.desc_old, true, stream))
        return st;
    if (remp_status st = launch_expand(*plan, *new_dev_tables, sh.new_block_size, nnz, new_tables->num_blocks,
                                       plan->new_live_blocks, ws, L.scan_new, L.desc_new, false, stream, L.bucket_new))
        return st;
    if (remp_status st = launch_sort_new(plan->new_live_blocks, new_tables->num_blocks, ws, L.desc_new, L.bucket_new,
                                         L.sorted_new, stream))
        return st;
    if (src->layout != kLayoutNHD || dst->layout != kLayoutNHD)
        return launch_local_tiles(*plan, items, src->layout, dst->layout, ws, stream);
    return launch_local(*plan, items, ws, stream);
}

}  // extern "C"
