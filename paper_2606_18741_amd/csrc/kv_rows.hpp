// Copies of whole paged rows split among several staging slices (copy_rows).
// Included by migrate.hip only (one translation unit holds every kernel).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kv_device.hpp"

namespace remp {

// ---------------------------------------------------------------------------
// whole paged rows
// ---------------------------------------------------------------------------
//
// When a new rank receives a layer's heads from several sources, the plain
// unpack writes each source's head range as its own pass over the new blocks,
// so every block row is opened once per source; likewise the plain pack reads
// an old block's rows once per destination when several destinations split
// its heads.  This variant takes one (layer, paged block, K/V) unit per
// workgroup and copies the unit's rows whole: each 16-byte vector of a row
// finds the staging slice holding its head and is read from (unpack) or
// written to (pack) that slice.  All layers of a call share the split of the
// row into slices.

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
    int32_t row_stride;       // full paged row (all local heads)
    int32_t block_size;
    int32_t nseg;
    int32_t head_bytes;
    uint32_t vpr_magic, vpr_shift;     // vectors per full row
    uint32_t unit_magic, unit_shift;   // vectors per (block, K/V) unit
    uint32_t vph_magic, vph_shift;     // vectors per head
    MergeSeg segs[kMaxMergeSegs];
    StampCheck check;
    uint64_t paged_k[kMaxMergeGroups];
    uint64_t paged_v[kMaxMergeGroups];
    uint64_t stage[kMaxMergeGroups][kMaxMergeSegs / 2];   // filled for nseg <= kMaxMergeSegs / 2
};
static_assert(sizeof(MergeArgs) < 4096, "whole-row kernel arguments must stay below 4 KiB");

template <int VEC, bool PACK, int THREADS, int UNROLL>
__global__ __launch_bounds__(THREADS) void copy_rows(const MergeArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_paged[kMaxUnitsPerWg];
    __shared__ int32_t s_tok[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ int32_t s_kv[kMaxUnitsPerWg];

    const bool stale = stamps_differ(args.check);   // acted on after the descriptor prologue
    uint32_t cx, cy;
    grid_cell<PACK ? kPackRowsXcd : kUnpackRowsXcd>(&cx, &cy);
    const int32_t g = static_cast<int32_t>(cy);
    const int32_t u0 = static_cast<int32_t>(cx) * args.units_per_wg;
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
    if (stale) {
        report_stale(args.check);
        return;
    }

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
                    const uint64_t stage = args.stage[g][sg] +
                                           static_cast<uint64_t>(s_kv[u]) * args.total_tokens * seg.row_bytes +
                                           static_cast<uint64_t>(s_tok[u] + row) * seg.row_bytes +
                                           static_cast<uint64_t>(h - seg.head0) * args.head_bytes +
                                           (c - h * vph) * VEC;
                    const uint64_t paged = s_paged[u] + static_cast<uint64_t>(row) * args.row_stride + c * VEC;
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

}  // namespace remp
