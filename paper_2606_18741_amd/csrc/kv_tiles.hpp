// Head-tile kernels through LDS for HND and ROCm pools: copy_tiles (pack / unpack)
// and copy_local_tiles (local copy between any layouts).
// Included by migrate.hip only (one translation unit holds every kernel).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kv_copy.hpp"     // kMaxLocalRows
#include "kv_device.hpp"

namespace remp {

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
    StampCheck check;
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

// Store the first `nbytes` bytes of a vector (whole elements of eb bytes) at a 16-byte aligned dst.
// The vector stays in registers: whole words first, then the elements of the last partial word.  Taking
// the vector's address instead (store_prefix_bytes) puts it in scratch memory on every pass of the
// caller's loop, also for whole vectors; in the head-tile unpack that cost 3-9% (MI355X, same process,
// ROCm pools: 7B MHA unpack +9.1% with this form, 70B GQA +3.0%, 13B MHA +3.2%).
__device__ __forceinline__ void store_prefix(const unsigned int __attribute__((ext_vector_type(4))) & val,
                                             void* dst, int32_t nbytes, int32_t eb) {
    unsigned int* o = reinterpret_cast<unsigned int*>(dst);
    const int32_t nw = nbytes >> 2;   // whole 4-byte words
    if (nw > 0) o[0] = val.x;
    if (nw > 1) o[1] = val.y;
    if (nw > 2) o[2] = val.z;
    if (nw > 3) o[3] = val.w;
    const int32_t rest = nbytes & 3;   // 2 (eb 2) or 1-3 (eb 1); eb 4 leaves none
    if (rest == 0) return;
    const unsigned int w = nw == 0 ? val.x : nw == 1 ? val.y : nw == 2 ? val.z : val.w;
    unsigned char* ob = reinterpret_cast<unsigned char*>(o + nw);
    if (eb == 2) {
        *reinterpret_cast<unsigned short*>(ob) = static_cast<unsigned short>(w);
    } else {
        ob[0] = static_cast<unsigned char>(w);
        if (rest > 1) ob[1] = static_cast<unsigned char>(w >> 8);
        if (rest > 2) ob[2] = static_cast<unsigned char>(w >> 16);
    }
}

// The same through the vector's bytes in memory.  The local head-tile copy keeps this form: with the
// register form its ROCm-pool local copies ran 1-3% slower (MI355X, same process, 13B MHA and 70B GQA
// shares), although both forms store the same bytes.
__device__ __forceinline__ void store_prefix_bytes(const unsigned int __attribute__((ext_vector_type(4))) & val,
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

    const bool stale = stamps_differ(args.check);   // acted on after the descriptor prologue
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
    if (stale) {
        report_stale(args.check);
        return;
    }

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


// Leading slots that have a source among the m (4, 8 or 16) consecutive one-byte flags at p (1: the
// row has a source), p aligned to m bytes: a ROCm V vector's slots in one or two LDS reads instead of
// one per slot.
__device__ __forceinline__ int32_t leading_sources(const uint8_t* p, int32_t m) {
    if (m == 4) {
        const uint32_t z = ~*reinterpret_cast<const uint32_t*>(p) & 0x01010101u;
        return z ? static_cast<int32_t>(__builtin_ctz(z) >> 3) : 4;
    }
    const uint64_t z0 = ~*reinterpret_cast<const uint64_t*>(p) & 0x0101010101010101ull;
    if (z0 || m == 8) return z0 ? static_cast<int32_t>(__builtin_ctzll(z0) >> 3) : 8;
    const uint64_t z1 = ~*reinterpret_cast<const uint64_t*>(p + 8) & 0x0101010101010101ull;
    return z1 ? 8 + static_cast<int32_t>(__builtin_ctzll(z1) >> 3) : 16;
}

// ---------------------------------------------------------------------------
// local copy between pools of any layouts (not both NHD), one head tile at a time
// ---------------------------------------------------------------------------
//
// A unit is one (new block, K or V, head of the slice) tile.  The prologue
// resolves each of its rows to the old (block, slot) through the old
// descriptors.  When both pools have the same layout, every 16-byte vector of
// a new tile has one 16-byte source vector in an old tile and is copied
// directly.  Otherwise the tile goes through LDS: phase 1 reads every live
// row's head vectors from the old pool in its layout into LDS (token-major;
// ROCm V tiles, where a token's elements of one head lie block_size elements
// apart, as vectors of m rows of one dim, stored element by element); phase 2
// writes the tile into the new pool in its layout, live slots only.

constexpr int kMaxLocalTileItems = 8;

// Dynamic LDS of copy_local_tiles: `tiles` head tiles of bn rows of lds_row bytes, then per row an
// 8-byte source base, a 4-byte slot and a 1-byte flag, then a 1-byte flag per tile.
inline int64_t local_tile_lds_bytes(int64_t tiles, int64_t bn, int64_t lds_row) {
    return tiles * bn * lds_row + tiles * bn * 13 + tiles;
}

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
    StampCheck check;
    LocalTileItem items[kMaxLocalTileItems];
};
static_assert(sizeof(LocalTileArgs) < 4096, "local tile kernel arguments must stay below 4 KiB");

__global__ __launch_bounds__(kTileThreads) void copy_local_tiles(const LocalTileArgs a) {
    typedef unsigned int V4 __attribute__((ext_vector_type(4)));
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    __shared__ uint64_t s_dst[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ int32_t s_kv[kMaxUnitsPerWg];

    if (stale_descriptors(a.check)) return;
    const LocalTileItem& it = a.items[blockIdx.y];
    const int32_t hc = it.heads;
    const int64_t ntiles = static_cast<int64_t>(a.n_new_desc) * 2 * hc;
    const int64_t g0 = static_cast<int64_t>(blockIdx.x) * a.tiles_per_wg;
    if (g0 >= ntiles) return;
    const int32_t nt = static_cast<int32_t>(min(static_cast<int64_t>(a.tiles_per_wg), ntiles - g0));
    const int tid = threadIdx.x;
    const int32_t bn = a.new_block_size, bo = a.old_block_size, hb = a.head_bytes, eb = a.elem_bytes;
    // per-(unit, row) arrays behind the tiles in the dynamic LDS, sized by the launch for tiles_per_wg
    // units (local_tile_lds_bytes), so that the workgroup holds only what its units need
    const uint32_t rows_cap = static_cast<uint32_t>(a.tiles_per_wg) * bn;
    unsigned char* rows_lds = lds + static_cast<uint32_t>(a.tiles_per_wg) * bn * static_cast<uint32_t>(a.lds_row);
    uint64_t* s_src = reinterpret_cast<uint64_t*>(rows_lds);               // old tile base of each row, 0: none
    int32_t* s_slot = reinterpret_cast<int32_t*>(rows_lds + rows_cap * 8);  // its old slot
    uint8_t* s_has = reinterpret_cast<uint8_t*>(rows_lds + rows_cap * 12);  // 1: the row has a source
    uint8_t* s_full = s_has + rows_cap;       // per tile, 1: every row live and with a source

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
        s_full[i] = nd.n == bn;
    }
    __syncthreads();
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
            // token within its sequence (negative when the device tables disagree: no source)
            const int32_t t = nd.tok - a.tok_off[nd.seq] + r;
            const int32_t ob = a.old_blk_off[nd.seq] + t / bo;
            slot = t - (t / bo) * bo;
            bool ok = t >= 0 && ob >= 0 && ob < a.n_old_desc;
            BlockDesc od{0, 0, 0, 0};
            if (ok) {
                od = a.old_desc[ob];
                ok = od.seq == nd.seq && slot < od.n;
            }
            if (ok)
                base = (kv ? it.src_v : it.src_k) + static_cast<uint64_t>(od.block) * a.old_block_stride +
                       static_cast<uint64_t>(j) * a.old_head_step;
            else
                *a.flag = kFlagTables;
        }
        s_src[x] = base;
        s_slot[x] = slot;
        s_has[x] = base != 0;
        if (base == 0) s_full[i] = 0;
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
            if (s_full[i]) {                                            // every vector of the tile is live
                __builtin_nontemporal_store(__builtin_nontemporal_load(src), dst);
            } else if (a.new_layout == kLayoutHND || s_kv[i] == 0) {
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
                const int32_t live = min(min(m, n - static_cast<int32_t>(s0)), leading_sources(s_has + i * bn + s0, m));
                if (live <= 0) continue;
                const V4 val = __builtin_nontemporal_load(src);
                if (live == m) __builtin_nontemporal_store(val, dst);
                else store_prefix_bytes(val, dst, live * eb, eb);
            }
        }
        return;
    }

    if (a.old_layout == a.new_layout) {
        // Same tile layout, block sizes that differ: token t of a sequence sits at row t mod bn of its new
        // block and at slot t mod bo of its old one, and both sizes are multiples of m (16 bytes of
        // elements), so a 16-byte vector of a new tile, part of one row (HND, ROCm K) or m rows of one dim
        // starting at a multiple of m (ROCm V), has one 16-byte source vector in an old tile: each is
        // copied directly, without LDS.  A V vector is read at its first row's source; one whose slot is
        // not a multiple of m (only when the device tables disagree with the host's) is not copied.
        for (uint32_t x = tid; x < total; x += kTileThreads) {
            const uint32_t i = fast_div(x, a.rows_magic, a.rows_shift);
            const uint32_t v = x - i * per_tile;
            const int32_t n = s_n[i];
            V4* dst = reinterpret_cast<V4*>(s_dst[i] + uint64_t(v) * 16);
            if (a.new_layout == kLayoutHND || s_kv[i] == 0) {
                uint32_t r;
                uint64_t off;                                            // within the old tile, but the slot
                uint32_t slot_bytes;
                if (a.new_layout == kLayoutHND) {                        // [slot][dim]
                    r = fast_div(v, a.vph_magic, a.vph_shift);
                    off = uint64_t(v - r * vph) * 16;
                    slot_bytes = static_cast<uint32_t>(hb);
                } else {                                                 // [dim / x][slot][x]
                    const uint32_t c = fast_div(v, a.bn_magic, a.bn_shift);
                    r = v - c * bn;
                    off = uint64_t(c) * bo * 16;
                    slot_bytes = 16;
                }
                if (static_cast<int32_t>(r) >= n || !s_has[i * bn + r]) continue;
                const uint64_t src = s_src[i * bn + r] + off + uint64_t(s_slot[i * bn + r]) * slot_bytes;
                __builtin_nontemporal_store(__builtin_nontemporal_load(reinterpret_cast<const V4*>(src)), dst);
            } else {                                                     // [dim][slot]
                const uint32_t e0 = v * m;
                const uint32_t dim = fast_div(e0, a.bn_magic, a.bn_shift);
                const uint32_t s0 = e0 - dim * bn;
                const int32_t live = min(min(m, n - static_cast<int32_t>(s0)), leading_sources(s_has + i * bn + s0, m));
                if (live <= 0) continue;
                const uint32_t slot = static_cast<uint32_t>(s_slot[i * bn + s0]);
                if (slot & static_cast<uint32_t>(m - 1)) continue;
                const V4 val = __builtin_nontemporal_load(reinterpret_cast<const V4*>(
                    s_src[i * bn + s0] + uint64_t(dim) * bo * eb + uint64_t(slot) * eb));
                if (live == m) __builtin_nontemporal_store(val, dst);
                else store_prefix_bytes(val, dst, live * eb, eb);
            }
        }
        return;
    }

    // phase 1: live rows of every tile from the old pool into LDS, token-major
    for (uint32_t x = tid; x < total; x += kTileThreads) {
        const uint32_t i = fast_div(x, a.rows_magic, a.rows_shift);
        const uint32_t rem = x - i * per_tile;
        if (a.old_layout == kLayoutRocmSplit && s_kv[i] == 1) {
            // [dim][slot] V tiles: vector rem holds m rows s0.. of one dim, whose old slots run on from a
            // multiple of m in one old block (as in the same-layout copy), so it is read as one 16-byte vector
            // at its first row's source and stored to LDS element by element; live rows outside that run
            // (only when the device tables disagree with the host's) are read element by element
            const uint32_t e0 = rem * m;
            const uint32_t dim = fast_div(e0, a.bn_magic, a.bn_shift);
            const uint32_t s0 = e0 - dim * bn;
            const int32_t nl = min(m, s_n[i] - static_cast<int32_t>(s0));    // live rows of the vector
            if (nl <= 0) continue;
            unsigned char* t0 = lds + i * tile_lds + s0 * lrow + dim * eb;
            const uint32_t slot0 = static_cast<uint32_t>(s_slot[i * bn + s0]);
            const int32_t run = (slot0 & static_cast<uint32_t>(m - 1)) ? 0 : leading_sources(s_has + i * bn + s0, m);
            if (run > 0)
                scatter_dim(__builtin_nontemporal_load(reinterpret_cast<const V4*>(
                                s_src[i * bn + s0] + uint64_t(dim) * bo * eb + uint64_t(slot0) * eb)),
                            t0, lrow, eb);
            for (int32_t k = run; k < nl; ++k) {
                const uint32_t row = s0 + static_cast<uint32_t>(k);
                if (!s_has[i * bn + row]) continue;
                const unsigned char* e = reinterpret_cast<const unsigned char*>(s_src[i * bn + row]) +
                                         uint64_t(dim) * bo * eb + uint64_t(s_slot[i * bn + row]) * eb;
                unsigned char* o = t0 + k * lrow;
                if (eb == 2) *reinterpret_cast<unsigned short*>(o) = *reinterpret_cast<const unsigned short*>(e);
                else if (eb == 4) *reinterpret_cast<unsigned int*>(o) = *reinterpret_cast<const unsigned int*>(e);
                else *o = *e;
            }
            continue;
        }
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
        } else {                                                         // [dim / x][slot][x] (K)
            val = __builtin_nontemporal_load(reinterpret_cast<const V4*>(base + uint64_t(c) * bo * 16 + slot * 16));
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
        const bool full = s_full[i];
        if (a.new_layout == kLayoutNHD) {
            const uint32_t r = fast_div(v, a.vph_magic, a.vph_shift);
            const uint32_t c = v - r * vph;
            if (full || (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0))
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + r * lrow + c * 16),
                                            reinterpret_cast<V4*>(s_dst[i] + uint64_t(r) * a.new_row_stride + c * 16));
            continue;
        }
        V4* dst = reinterpret_cast<V4*>(s_dst[i] + uint64_t(v) * 16);
        if (a.new_layout == kLayoutHND) {
            const uint32_t r = fast_div(v, a.vph_magic, a.vph_shift);
            if (full || (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0))
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + r * lrow + (v - r * vph) * 16), dst);
        } else if (s_kv[i] == 0) {                                       // [dim / x][slot][x]
            const uint32_t c = fast_div(v, a.bn_magic, a.bn_shift);
            const uint32_t r = v - c * bn;
            if (full || (static_cast<int32_t>(r) < n && s_src[i * bn + r] != 0))
                __builtin_nontemporal_store(*reinterpret_cast<const V4*>(tl + r * lrow + c * 16), dst);
        } else {                                                         // [dim][slot]
            const uint32_t e0 = v * m;
            const uint32_t dim = fast_div(e0, a.bn_magic, a.bn_shift);
            const uint32_t s0 = e0 - dim * bn;
            // rows without a source stay untouched
            const int32_t live =
                full ? m : min(min(m, n - static_cast<int32_t>(s0)), leading_sources(s_has + i * bn + s0, m));
            if (live <= 0) continue;
            const V4 val = gather_dim(tl + s0 * lrow + dim * eb, lrow, eb);
            if (live == m) __builtin_nontemporal_store(val, dst);
            else store_prefix_bytes(val, dst, live * eb, eb);
        }
    }
}

}  // namespace remp
