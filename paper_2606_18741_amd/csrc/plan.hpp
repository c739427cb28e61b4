// Internal plan representation shared by the host planner and the launch code.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "remp_kv.h"

namespace remp {

// One send/receive item of the plan: old rank `src` ships heads
// [head_begin, head_begin + head_count) of layer `layer` to new rank `dst`.
struct Item {
    int32_t src, dst, layer, head_begin, head_count;
    int32_t pair;        // index into Plan::pairs
};

struct Pair {
    int32_t src, dst;
    int32_t layer_begin, layer_end;
    int32_t head_begin, head_count;
    int64_t slice_bytes;
};

// Ownership of one topology (Section 3.4.1).  Layers: stage p holds
// [starts[p], starts[p+1]) (by default equal ranges [p*L/PP, (p+1)*L/PP)).
// Heads: with TP <= H, tensor rank t holds
// [t*H/TP, (t+1)*H/TP); with TP > H (TP a multiple of H, GQA replication) it
// holds the single head t*H/TP, and each head has TP/H replicas.
struct Ownership {
    int32_t tp = 1, pp = 1, L = 0, H = 0;
    std::vector<int32_t> starts;          // [pp + 1] stage boundaries
    std::vector<int32_t> stage_of_layer;  // [L]
    void set_layers(const int32_t* layer_starts) {
        starts.resize(pp + 1);
        for (int32_t p = 0; p <= pp; ++p)
            starts[p] = layer_starts ? layer_starts[p] : static_cast<int32_t>(static_cast<int64_t>(p) * L / pp);
        stage_of_layer.assign(L, 0);
        for (int32_t p = 0; p < pp; ++p)
            for (int32_t l = starts[p]; l < starts[p + 1]; ++l) stage_of_layer[l] = p;
    }
    int32_t layers_of_rank(int32_t r) const { return starts[stage_of(r) + 1] - starts[stage_of(r)]; }
    int32_t heads_per_rank() const { return tp <= H ? H / tp : 1; }
    int32_t replicas() const { return tp <= H ? 1 : tp / H; }
    int32_t pp_owner(int32_t l) const { return stage_of_layer[l]; }
    int32_t rank(int32_t stage, int32_t t) const { return stage * tp + t; }
    int32_t stage_of(int32_t r) const { return r / tp; }
    int32_t tp_of(int32_t r) const { return r % tp; }
    int32_t first_layer(int32_t r) const { return starts[stage_of(r)]; }
    int32_t first_head_of_tp(int32_t t) const { return static_cast<int32_t>(static_cast<int64_t>(t) * H / tp); }
    int32_t first_head(int32_t r) const { return first_head_of_tp(tp_of(r)); }
    // replica index of tensor rank t among the ranks holding its head (0 without replication)
    int32_t replica_index(int32_t t) const { return tp <= H ? 0 : t % (tp / H); }
    // tensor rank holding head h as replica k
    int32_t tp_of_head(int32_t h, int32_t k) const { return tp <= H ? h / (H / tp) : h * (tp / H) + k; }
    int32_t world() const { return tp * pp; }
};

}  // namespace remp

struct remp_kv_plan_s {
    remp_topo old_topo, new_topo;
    remp_kv_shape shape;
    remp::Ownership own_old, own_new;
    int32_t num_seqs = 0;
    std::vector<int32_t> seq_lens;
    std::vector<int32_t> old_row_offsets;
    std::vector<int32_t> old_block_ids;
    int64_t old_num_blocks = 0;
    int64_t old_nnz = 0;
    int64_t total_tokens = 0;
    int64_t old_live_blocks = 0;
    int64_t new_live_blocks = 0;
    std::vector<remp::Item> items;     // Algorithm 1 order: layer, then new tensor rank, then old tensor rank
    std::vector<remp::Pair> pairs;     // ordered by (src, dst)
    std::vector<int32_t> pair_index;   // [old_world * new_world] -> pair or -1
    uint64_t serial = 0;               // unique per plan in the process (descriptor stamps)
    int64_t wg_bytes = 0;              // tuning hook REMP_KV_WG_BYTES, read once at plan creation (0: built-in)
};

namespace remp {

// Thread-local error reporting shared by every entry point.
remp_status fail(remp_status st, const std::string& msg);
void clear_error();

int64_t ceil_div(int64_t a, int64_t b);

// Byte offsets inside the caller's workspace.  A 256-byte header holds the
// status flag (int32 at 0) and the stamps of the old and the new descriptors
// (uint64 at stamp_old and stamp_new: which plan and tables the descriptors
// were expanded from, so a later call may reuse them).  Each scan area holds
// token and block offsets per sequence ([S+1] int32 each); each descriptor
// area holds one 16-byte descriptor per live block.  Pack uses the old areas,
// unpack the new ones, the local copy both.  The new descriptors are also
// bucket-sorted by physical block (bucket counters, then the sorted copy) so
// that the unpack side writes the paged pool in ascending address order.
struct WorkspaceLayout {
    int64_t stamp_old, stamp_new;
    int64_t scan_old, scan_new, desc_old, desc_new, bucket_new, sorted_new, total;
};
WorkspaceLayout workspace_layout(const remp_kv_plan_t& p);
int64_t workspace_bytes(const remp_kv_plan_t& p);
const Pair* find_pair(const remp_kv_plan_t& p, int32_t src, int32_t dst);

}  // namespace remp
