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
// workgroup and copies the whole unit: the row is split into nseg equal
// shares (one per staging slice, consecutive heads), and the workgroup copies
// share 0 of all the unit's rows, then share 1, and so on, so every slice's
// part of the unit is one contiguous staging range read (unpack) or written
// (pack) in order, while the paged block is covered whole by one workgroup.
// All layers of a call share the split of the row into slices.

constexpr int kMaxMergeSegs = 4;     // slices per row
constexpr int kMaxMergeGroups = 8;   // layers per launch

struct MergeArgs {
    const BlockDesc* desc;
    int64_t block_stride;
    int64_t total_tokens;
    int32_t n_desc;
    int32_t units_per_wg;
    int32_t row_stride;       // full paged row (all local heads)
    int32_t block_size;
    int32_t nseg;             // shares per row
    uint32_t seg_bytes;       // bytes of one share of a row (= row_stride / nseg)
    uint32_t unit_magic, unit_shift;   // division by vectors per (block, K/V) unit
    uint32_t seg_magic, seg_shift;     // division by vectors per share of a unit (block_size * share vectors)
    uint32_t vps_magic, vps_shift;     // division by vectors per share of a row
    StampCheck check;
    uint64_t paged_k[kMaxMergeGroups];
    uint64_t paged_v[kMaxMergeGroups];
    uint64_t stage[kMaxMergeGroups][kMaxMergeSegs];
};
static_assert(sizeof(MergeArgs) < 4096, "whole-row kernel arguments must stay below 4 KiB");

template <int VEC, bool PACK, int THREADS, int UNROLL, bool XCD>
__global__ __launch_bounds__(THREADS) void copy_rows(const MergeArgs args) {
    typedef typename VecT<VEC>::type V;
    __shared__ uint64_t s_paged[kMaxUnitsPerWg];
    __shared__ int32_t s_tok[kMaxUnitsPerWg];
    __shared__ int32_t s_n[kMaxUnitsPerWg];
    __shared__ int32_t s_kv[kMaxUnitsPerWg];

    const bool stale = stamps_differ(args.check);   // acted on after the descriptor prologue
    uint32_t cx, cy;
    grid_cell<XCD>(&cx, &cy);
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

    // the group's staging bases, uniform: each lane selects its share's base (a per-lane index into the
    // argument array would load it from memory inside the loop and serialise the vector loads)
    const uint64_t st0 = args.stage[g][0], st1 = args.stage[g][1], st2 = args.stage[g][2], st3 = args.stage[g][3];
    const uint32_t vps = args.seg_bytes / VEC;                         // vectors per share of a row
    const uint32_t per_seg = static_cast<uint32_t>(args.block_size) * vps;
    const uint32_t unit = static_cast<uint32_t>(args.nseg) * per_seg;
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
                // idx = ((unit, share), row, vector of the share)
                const uint32_t u = fast_div(idx, args.unit_magic, args.unit_shift);
                const uint32_t rem = idx - u * unit;
                const uint32_t sg = fast_div(rem, args.seg_magic, args.seg_shift);
                const uint32_t r2 = rem - sg * per_seg;
                const uint32_t row = fast_div(r2, args.vps_magic, args.vps_shift);
                const uint32_t cs = r2 - row * vps;
                if (static_cast<int32_t>(row) < s_n[u]) {
                    const uint64_t base = sg == 0 ? st0 : sg == 1 ? st1 : sg == 2 ? st2 : st3;
                    const uint64_t stage = base +
                                           static_cast<uint64_t>(s_kv[u]) * args.total_tokens * args.seg_bytes +
                                           static_cast<uint64_t>(s_tok[u] + row) * args.seg_bytes + cs * VEC;
                    const uint64_t paged = s_paged[u] + static_cast<uint64_t>(row) * args.row_stride +
                                           (sg * vps + cs) * VEC;
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
