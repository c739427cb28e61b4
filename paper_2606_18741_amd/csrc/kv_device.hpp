// Device data structures and launch constants of the KV-migration kernels.
// Included by migrate.hip only (one translation unit holds every kernel).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

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

// Values of the workspace status flag (int32 at byte 0 of the workspace).
constexpr int32_t kFlagTables = 1;   // the device tables would have indexed out of range
constexpr int32_t kFlagStale = 2;    // a reusing call found descriptors of other tables

// Check of reused descriptors.  A call that expands its own descriptors passes
// at[] = NULL; a call that reuses them names the stamps they must carry (one
// per side it reads: old and new).  On a mismatch every workgroup leaves
// before it writes anything outside LDS, and the first one sets the flag.
// Kernels whose prologue only reads the descriptor array itself test the
// result after that prologue (the stamp load then overlaps the descriptor
// loads); kernels that follow a descriptor to other arrays test it first.
struct StampCheck {
    const uint64_t* at[2];
    uint64_t want[2];
    int32_t* flag;
};

__device__ __forceinline__ bool stamps_differ(const StampCheck& c) {
    bool differ = false;
#pragma unroll
    for (int i = 0; i < 2; ++i)
        if (c.at[i] && *c.at[i] != c.want[i]) differ = true;
    return differ;
}

__device__ __forceinline__ void report_stale(const StampCheck& c) {
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *c.flag = kFlagStale;
}

__device__ __forceinline__ bool stale_descriptors(const StampCheck& c) {
    if (!stamps_differ(c)) return false;
    report_stale(c);
    return true;
}

// Whole paged rows (copy_rows) when several staging slices split every row into
// equal shares: unpack when several sources fill a new rank's rows (shares of at
// least 256 B), pack when several destinations split an old rank's rows into
// 256 B shares.  A/B on MI355X against per-slice copies (one process, memory
// prewarmed, three repetitions): unpack 70B GQA (two 256 B shares) -1.6% time,
// 7B (two 2 KiB) -2.8%; pack long context (two 256 B) -4%, but 13B (two 2.5 KiB)
// +1% and DeepSeek-32B (four 512 B) +4%, in either order inside the unit and
// with or without the XCD cell order: whole rows pay on the pack side only where
// the per-slice pack would read 256 B fragments of each row.  Inside a unit each
// share's rows are copied in turn (segment-major); cells in plain order.
constexpr bool kMergeRows = true;
constexpr bool kPackRows = true;
constexpr uint32_t kUnpackRowsMinShareBytes = 256;
constexpr uint32_t kPackRowsMinShareBytes = 256;
constexpr uint32_t kPackRowsMaxShareBytes = 256;
constexpr uint32_t kUnpackRowsMaxShareBytes = 0xFFFFFFFFu;
// Small whole-row units (the 70B GQA unpack: 8 KiB) run one unit per 256-thread workgroup, two vectors
// per lane (A/B on MI355X against 128 x 4: 70B unpack -1.0%; 512 x 1 and 64 x 8 slower).
constexpr int kRowsSmallThreads = 256, kRowsSmallUnroll = 2;
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
// Unpack workgroups that move at most 4 KiB (one 4 KiB unit, as with one 256-byte head row per token
// at 16 tokens per block) run one wave of 4 vectors per lane, so no lane idles (A/B on MI355X, one
// process, Qwen3-30B-A3B share: unpack +2.5%; with 8 KiB units the 128-thread shape stays faster).
constexpr int kUnpackTinyThreads = 64;
constexpr int64_t kUnpackTinyWgBytes = 4 * 1024;
constexpr int kPackSmallThreads = 64, kPackSmallUnroll = 4;   // pack of small units: one wave per unit
// Pack of small units that take part of each row (the old rank's heads split among several new ranks,
// e.g. 512 of 2048 bytes at TP1 -> TP4): four waves per unit with one vector per lane (A/B on MI355X,
// one process, DeepSeek-32B share TP1/PP8 -> TP4/PP2: pack +3.7%; whole-row units stay faster with
// one wave: 70B GQA -2.9%, Qwen3-30B-A3B -1.1% with this shape).
constexpr int kPackPartialThreads = 256, kPackPartialUnroll = 1;
// XCD-contiguous cell order, per launch kind (A/B on MI355X, one process: with it, 7B MHA pack
// +5%; 70B GQA small-unit pack -1.5% and unpack of block-sorted descriptors -1.6%)
constexpr bool kPackSmallXcd = false;
constexpr bool kUnpackSmallXcd = false;
constexpr bool kPackLargeXcd = true;
constexpr bool kUnpackLargeXcd = true;
// The same order for large-unit whole-row copies and local copies (MI355X, one process, three
// repetitions): 7B MHA whole-row unpack -1.9%, copy_local -6.4% (7B) and -2.6% (13B MHA).
constexpr bool kRowsLargeXcd = true;
constexpr bool kLocalLargeXcd = true;
constexpr int64_t kSmallWgBytes = 4 * 1024;
// The local copy's per-unit prologue (three dependent descriptor reads) wants several units per
// workgroup: 16 KiB against 8 KiB, copy_local alone on MI355X (one process, memory prewarmed):
// 70B GQA -4.7% time, long context -5.8%, Qwen3-30B-A3B -5.6% (DeepSeek-32B -3.6% without the
// prewarm); 256 x 4 or 32 KiB were slower (8 KiB against 4 KiB had been +14%).
constexpr int64_t kLocalSmallWgBytes = 16 * 1024;
// and 256 threads with two loads in flight per lane (one process, five repetitions, against 128 x 4):
// 70B GQA -2.3% time, long context -1.1%, Qwen3-30B-A3B -2.0%, DeepSeek-32B +0.4%; 512 x 1, and 256 x 2
// with 8 or 32 KiB per workgroup, were 3-9% slower than 128 x 4.
constexpr int kLocalSmallThreads = 256, kLocalSmallUnroll = 2;
// Large units (MHA rows of 2 KiB and more): 16-wave workgroups with two loads in flight per lane,
// against 4 waves with eight (MI355X, one process, three repetitions): 7B MHA step -3.4%, 13B MHA
// pack -2.1% and unpack -2.9% time.  The local copy's optimum differs: 512 x 4 was faster than
// 256 x 8 on both shapes (7B -4%, 13B -2.8%), 1024 x 2 -10.7% on 7B but +0.8% on 13B.
constexpr int kLargeThreads = 1024, kLargeUnroll = 2;
constexpr int kLocalLargeThreads = 512, kLocalLargeUnroll = 4;
// and at most 32 KiB per workgroup (7B MHA copy_local -5% against 64 KiB; 13B MHA, whose 40 KiB units
// go one per workgroup either way, unchanged)
constexpr int64_t kLocalLargeWgBytes = 32 * 1024;
constexpr int64_t kLargeWgBytes = 64 * 1024;
constexpr int kScanThreads = 1024;

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
    StampCheck check;
    CopyItem items[kMaxItems];
};
static_assert(sizeof(CopyArgs) < 4096, "copy kernel arguments must stay below 4 KiB");

}  // namespace remp
