// The pack / unpack copy kernel (copy_slices) and the NHD local copy (copy_local).
// Included by migrate.hip only (one translation unit holds every kernel).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kv_device.hpp"

namespace remp {

// ---------------------------------------------------------------------------
// pack / unpack copy
// ---------------------------------------------------------------------------


// CHECK: the call reuses descriptors, so their stamps are compared (the calls
// that expand their own descriptors run the variant without the comparison).
template <int VEC, bool PACK, int THREADS, int UNROLL, bool XCD, bool CHECK>
__global__ __launch_bounds__(THREADS) void copy_slices(const CopyArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_paged[kMaxUnitsPerWg];
    __shared__ uint64_t s_stage[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];

    const bool stale = CHECK && stamps_differ(args.check);   // acted on after the descriptor prologue
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
    if (CHECK && stale) {
        report_stale(args.check);
        return;
    }

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
    StampCheck check;
    LocalItem items[kMaxLocalItems];
};
static_assert(sizeof(LocalArgs) < 4096, "local copy kernel arguments must stay below 4 KiB");

template <int VEC, int THREADS, int UNROLL, bool XCD>
__global__ __launch_bounds__(THREADS) void copy_local(const LocalArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_dst[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ uint64_t s_src[kMaxLocalRows];

    if (stale_descriptors(args.check)) return;
    uint32_t cx, cy;
    grid_cell<XCD>(&cx, &cy);
    const LocalItem& it = args.items[cy];
    const int32_t u0 = static_cast<int32_t>(cx) * args.units_per_wg;
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
            // token within its sequence: the new expansion's token offset less the old one's, so
            // device tables that disagree can make it negative; such a row has no source
            const int32_t t = d.tok - args.tok_off[d.seq] + r;
            const int32_t ob = args.old_blk_off[d.seq] + t / bo;
            const int32_t slot = t - (t / bo) * bo;
            bool ok = t >= 0 && ob >= 0 && ob < args.n_old_desc;
            BlockDesc od{0, 0, 0, 0};
            if (ok) {
                od = args.old_desc[ob];
                ok = od.seq == d.seq && slot < od.n;
            }
            if (ok)
                a = ((g & 1) ? it.src_v : it.src_k) + static_cast<uint64_t>(od.block) * args.old_block_stride +
                    static_cast<uint64_t>(slot) * args.old_row_stride;
            else
                *args.flag = kFlagTables;
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

}  // namespace remp
