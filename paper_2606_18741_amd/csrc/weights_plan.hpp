// Internal representation of a weight-shard plan (host store -> GPU shards).
#pragma once

#include <cstdint>
#include <vector>

#include "remp_weights.h"

namespace remp {

struct WPart {
    const char* host;
    int64_t rows, cols;
    int32_t split, units;
};

struct WTensor {
    int32_t layer;
    int32_t first_part, num_parts;
    int64_t shard_cols;   // the same for every tensor rank
};

// One rectangular piece of a shard: `rows` rows of `width` bytes, read at
// `src_off` bytes into part `part` of the store with a row pitch of `pitch`
// bytes, written contiguously at `dst_off` bytes into the shard.
struct WSeg {
    int32_t part;
    int64_t src_off, pitch, width, rows, dst_off;
};

}  // namespace remp

struct remp_w_plan_s {
    int32_t tp = 1, pp = 1, num_layers = 0, elem_bytes = 0;
    std::vector<int32_t> starts;          // [pp + 1] stage boundaries
    std::vector<int32_t> stage_of_layer;  // [num_layers]
    std::vector<remp::WTensor> tensors;
    std::vector<remp::WPart> parts;
};

namespace remp {

// Units [u0, u0 + n) of a part split into `units` that tensor rank t keeps
// under TP (Section 3.3, tensor slicing by the target tensor-parallel degree).
void w_unit_range(int32_t t, int32_t tp, int32_t units, int32_t* u0, int32_t* n);

// Whether pipeline stage `stage` holds tensor `w` (its layer's stage, or the
// first / last stage for tensors outside the decoder layers).
bool w_holds(const remp_w_plan_t& p, int32_t stage, const WTensor& w);

// Shard rows of `part` on tensor rank t.
int64_t w_part_rows(const remp_w_plan_t& p, const WPart& part, int32_t t);

// Append the segments of tensor `tensor` on `rank` (none if not held).
void w_segments(const remp_w_plan_t& p, int32_t rank, int32_t tensor, std::vector<WSeg>& out);

}  // namespace remp
