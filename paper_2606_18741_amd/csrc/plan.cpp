// Host planner: ownership functions, migration-plan construction and validation.
//
// ReMP Section 3.4.1 defines ownership by two functions, pp_owner(l, PP) and
// tp_owner(h, TP), composed into a global rank; Section 3.4.2 (Algorithm 1)
// builds the plan by intersecting, layer by layer, the head range each new
// tensor rank needs with the head range each old tensor rank holds.  Every
// non-empty intersection is one item, seen by the old rank as a send and by
// the new rank as a receive.  The plan carries no device memory.
#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <new>
#include <string>

#include "plan.hpp"

namespace remp {

static thread_local std::string g_last_error;

remp_status fail(remp_status st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

void clear_error() { g_last_error.clear(); }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

const Pair* find_pair(const remp_kv_plan_t& p, int32_t src, int32_t dst) {
    if (src < 0 || dst < 0 || src >= p.own_old.world() || dst >= p.own_new.world()) return nullptr;
    int32_t i = p.pair_index[static_cast<size_t>(src) * p.own_new.world() + dst];
    return i < 0 ? nullptr : &p.pairs[i];
}

static int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

// Workspace: [header: flag, descriptor stamps; 256 B][old scan][new scan][old descriptors]
// [new descriptors][bucket counters][sorted new descriptors], each area 256-aligned.
WorkspaceLayout workspace_layout(const remp_kv_plan_t& p) {
    WorkspaceLayout w;
    w.stamp_old = 8;
    w.stamp_new = 16;
    const int64_t scan = align256(2 * (static_cast<int64_t>(p.num_seqs) + 1) * 4);
    w.scan_old = 256;
    w.scan_new = w.scan_old + scan;
    w.desc_old = w.scan_new + scan;
    w.desc_new = w.desc_old + align256(std::max<int64_t>(p.old_live_blocks, 1) * 16);
    w.bucket_new = w.desc_new + align256(std::max<int64_t>(p.new_live_blocks, 1) * 16);
    w.sorted_new = w.bucket_new + align256(std::max<int64_t>(p.new_live_blocks, 1) * 4);
    w.total = w.sorted_new + align256(std::max<int64_t>(p.new_live_blocks, 1) * 16);
    return w;
}

int64_t workspace_bytes(const remp_kv_plan_t& p) { return workspace_layout(p).total; }

static remp_status check_topo(const remp_topo* t, const char* which, const remp_kv_shape& s) {
    if (!t) return fail(REMP_E_INVALID, std::string(which) + " topology is NULL");
    if (t->tp < 1 || t->pp < 1)
        return fail(REMP_E_INVALID, std::string(which) + " topology needs TP >= 1 and PP >= 1");
    if (t->pp > s.num_layers)
        return fail(REMP_E_INVALID, std::string(which) + " topology has more pipeline stages than layers");
    if (s.num_kv_heads % t->tp != 0 && t->tp % s.num_kv_heads != 0)
        return fail(REMP_E_UNSUPPORTED, std::string(which) + " TP=" + std::to_string(t->tp) +
                                            " neither divides nor is a multiple of num_kv_heads=" +
                                            std::to_string(s.num_kv_heads));
    if (t->layer_starts) {
        if (t->layer_starts[0] != 0 || t->layer_starts[t->pp] != s.num_layers)
            return fail(REMP_E_INVALID, std::string(which) + " layer_starts must run from 0 to num_layers");
        for (int32_t p = 0; p < t->pp; ++p)
            if (t->layer_starts[p + 1] <= t->layer_starts[p])
                return fail(REMP_E_INVALID, std::string(which) + " layer_starts must increase (every stage holds a layer)");
        return REMP_OK;
    }
    if (s.num_layers % t->pp != 0)
        return fail(REMP_E_UNSUPPORTED, std::string(which) + " PP=" + std::to_string(t->pp) +
                                            " does not divide num_layers=" + std::to_string(s.num_layers) +
                                            " (give layer_starts for an uneven split)");
    return REMP_OK;
}

}  // namespace remp

using namespace remp;

extern "C" {

remp_status remp_kv_plan(const remp_topo* old_topo, const remp_topo* new_topo, const remp_kv_shape* shape,
                         const remp_block_tables* old_tables, remp_kv_plan_t** out) {
    clear_error();
    if (!out) return fail(REMP_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!shape) return fail(REMP_E_INVALID, "shape is NULL");
    const remp_kv_shape s = *shape;
    if (s.num_layers < 1 || s.num_kv_heads < 1 || s.head_dim < 1 || s.old_block_size < 1 ||
        s.new_block_size < 1)
        return fail(REMP_E_INVALID, "shape sizes must be positive");
    if (s.elem_bytes != 1 && s.elem_bytes != 2 && s.elem_bytes != 4)
        return fail(REMP_E_INVALID, "elem_bytes must be 1, 2 or 4");
    if (static_cast<int64_t>(s.num_kv_heads) * s.head_dim * s.elem_bytes > (int64_t(1) << 30))
        return fail(REMP_E_UNSUPPORTED, "a token row of all heads exceeds 1 GiB");
    if (remp_status st = check_topo(old_topo, "old", s)) return st;
    if (remp_status st = check_topo(new_topo, "new", s)) return st;
    if (!old_tables) return fail(REMP_E_INVALID, "old_tables is NULL");
    const remp_block_tables& t = *old_tables;
    if (t.num_seqs < 0) return fail(REMP_E_INVALID, "num_seqs < 0");
    if (t.num_seqs > 0 && (!t.seq_lens || !t.row_offsets))
        return fail(REMP_E_INVALID, "old_tables arrays are NULL");
    if (t.num_blocks < 0 || t.num_blocks > std::numeric_limits<int32_t>::max())
        return fail(REMP_E_INVALID, "old_tables.num_blocks must be in [0, 2^31)");

    remp_kv_plan_t* p = new (std::nothrow) remp_kv_plan_t();
    if (!p) return fail(REMP_E_INVALID, "out of host memory");
    static std::atomic<uint64_t> next_serial{1};
    p->serial = next_serial.fetch_add(1);
    if (const char* wg = std::getenv("REMP_KV_WG_BYTES")) {   // tuning hook, see remp_kv.h
        const long long v = std::atoll(wg);
        p->wg_bytes = v > 0 ? std::min<long long>(v, int64_t(1) << 30) : 0;
    }
    p->old_topo = *old_topo;
    p->new_topo = *new_topo;
    p->shape = s;
    p->own_old.tp = old_topo->tp;
    p->own_old.pp = old_topo->pp;
    p->own_old.L = s.num_layers;
    p->own_old.H = s.num_kv_heads;
    p->own_old.set_layers(old_topo->layer_starts);
    p->own_new.tp = new_topo->tp;
    p->own_new.pp = new_topo->pp;
    p->own_new.L = s.num_layers;
    p->own_new.H = s.num_kv_heads;
    p->own_new.set_layers(new_topo->layer_starts);
    p->num_seqs = t.num_seqs;
    p->old_num_blocks = t.num_blocks;

    // --- old tables: structure, lengths, ids ---------------------------------
    int64_t nnz = 0;
    if (t.num_seqs > 0) {
        if (t.row_offsets[0] < 0) {
            delete p;
            return fail(REMP_E_INVALID, "row_offsets[0] < 0");
        }
        nnz = t.row_offsets[t.num_seqs];
        if (nnz > 0 && !t.block_ids) {
            delete p;
            return fail(REMP_E_INVALID, "old block_ids is NULL");
        }
    }
    p->seq_lens.assign(t.seq_lens, t.seq_lens + t.num_seqs);
    p->old_row_offsets.assign(t.row_offsets, t.row_offsets + (t.num_seqs > 0 ? t.num_seqs + 1 : 0));
    if (t.num_seqs == 0) p->old_row_offsets.assign(1, 0);
    p->old_block_ids.assign(t.block_ids ? t.block_ids : nullptr, t.block_ids ? t.block_ids + nnz : nullptr);
    p->old_nnz = nnz;
    int64_t T = 0, nb_old = 0, nb_new = 0;
    for (int32_t q = 0; q < t.num_seqs; ++q) {
        int32_t n = p->seq_lens[q];
        int32_t a = p->old_row_offsets[q], b = p->old_row_offsets[q + 1];
        if (n < 0) {
            delete p;
            return fail(REMP_E_INVALID, "seq_lens[" + std::to_string(q) + "] < 0");
        }
        if (b < a) {
            delete p;
            return fail(REMP_E_INVALID, "row_offsets decrease at sequence " + std::to_string(q));
        }
        int64_t need = ceil_div(n, s.old_block_size);
        if (b - a < need) {
            delete p;
            return fail(REMP_E_INVALID, "old table row of sequence " + std::to_string(q) + " has " +
                                            std::to_string(b - a) + " entries, needs " + std::to_string(need));
        }
        for (int64_t j = 0; j < need; ++j) {
            int32_t id = p->old_block_ids[a + j];
            if (id < 0 || id >= t.num_blocks) {
                delete p;
                return fail(REMP_E_RANGE, "old block id " + std::to_string(id) + " (sequence " + std::to_string(q) +
                                              ") outside [0, " + std::to_string(t.num_blocks) + ")");
            }
        }
        T += n;
        nb_old += need;
        nb_new += ceil_div(n, s.new_block_size);
    }
    if (T > std::numeric_limits<int32_t>::max()) {
        delete p;
        return fail(REMP_E_UNSUPPORTED, "more than 2^31 - 1 live tokens");
    }
    // launch grids index (block, K/V) units of up to 8 slices with 32-bit workgroup ids
    if (nb_old >= (int64_t(1) << 28) || nb_new >= (int64_t(1) << 28)) {
        delete p;
        return fail(REMP_E_UNSUPPORTED, "2^28 or more live blocks");
    }
    p->total_tokens = T;
    p->old_live_blocks = nb_old;
    p->new_live_blocks = nb_new;

    // --- Algorithm 1: per layer, each new tensor rank's head range against the
    // old tensor ranks' ranges; every non-empty overlap is one item.  When old
    // heads are replicated (TP_old > H) several old ranks hold the same head and
    // one of them is the source: the destination itself if it holds a replica
    // (a local copy), else replica (new replica index mod old replicas), which
    // spreads the sends over the replicas.
    const Ownership& O = p->own_old;
    const Ownership& N = p->own_new;
    const int64_t row = static_cast<int64_t>(s.head_dim) * s.elem_bytes;
    p->pair_index.assign(static_cast<size_t>(O.world()) * N.world(), -1);
    for (int32_t l = 0; l < s.num_layers; ++l) {
        const int32_t old_stage = O.pp_owner(l), new_stage = N.pp_owner(l);
        for (int32_t ntp = 0; ntp < N.tp; ++ntp) {
            const int32_t t0 = N.first_head_of_tp(ntp), t1 = t0 + N.heads_per_rank();
            const int32_t dst = N.rank(new_stage, ntp);
            if (O.replicas() == 1) {
                for (int32_t otp = 0; otp < O.tp; ++otp) {
                    const int32_t s0 = O.first_head_of_tp(otp), s1 = s0 + O.heads_per_rank();
                    const int32_t h0 = std::max(t0, s0), h1 = std::min(t1, s1);
                    if (h0 >= h1) continue;
                    p->items.push_back(Item{O.rank(old_stage, otp), dst, l, h0, h1 - h0, -1});
                }
                continue;
            }
            // replicated old heads: one old head per old rank, choose a replica per target head
            for (int32_t h = t0; h < t1; ++h) {
                int32_t otp = -1;
                for (int32_t k = 0; k < O.replicas(); ++k)
                    if (O.rank(old_stage, O.tp_of_head(h, k)) == dst) otp = O.tp_of_head(h, k);
                if (otp < 0) otp = O.tp_of_head(h, N.replica_index(ntp) % O.replicas());
                p->items.push_back(Item{O.rank(old_stage, otp), dst, l, h, 1, -1});
            }
        }
    }
    // group items into pairs; within a pair the layers form one range and the heads are fixed
    std::vector<std::vector<int32_t>> by_pair(static_cast<size_t>(O.world()) * N.world());
    for (size_t i = 0; i < p->items.size(); ++i)
        by_pair[static_cast<size_t>(p->items[i].src) * N.world() + p->items[i].dst].push_back(static_cast<int32_t>(i));
    for (int32_t src = 0; src < O.world(); ++src) {
        for (int32_t dst = 0; dst < N.world(); ++dst) {
            auto& v = by_pair[static_cast<size_t>(src) * N.world() + dst];
            if (v.empty()) continue;
            const Item& first = p->items[v.front()];
            Pair pr{src, dst, first.layer, first.layer + 1, first.head_begin, first.head_count, 0};
            for (size_t k = 1; k < v.size(); ++k) {
                const Item& it = p->items[v[k]];
                if (it.layer != pr.layer_end || it.head_begin != pr.head_begin || it.head_count != pr.head_count) {
                    delete p;
                    return fail(REMP_E_INVALID, "internal: pair slices are not a layer range with fixed heads");
                }
                pr.layer_end = it.layer + 1;
            }
            pr.slice_bytes = 2 * T * pr.head_count * row;
            p->pair_index[static_cast<size_t>(src) * N.world() + dst] = static_cast<int32_t>(p->pairs.size());
            for (int32_t k : v) p->items[k].pair = static_cast<int32_t>(p->pairs.size());
            p->pairs.push_back(pr);
        }
    }
    *out = p;
    return REMP_OK;
}

void remp_kv_plan_destroy(remp_kv_plan_t* plan) { delete plan; }

remp_status remp_kv_plan_get_info(const remp_kv_plan_t* plan, remp_kv_plan_info* out) {
    clear_error();
    if (!plan || !out) return fail(REMP_E_INVALID, "plan or out is NULL");
    out->old_world = plan->own_old.world();
    out->new_world = plan->own_new.world();
    out->num_pairs = static_cast<int32_t>(plan->pairs.size());
    out->num_items = static_cast<int32_t>(plan->items.size());
    out->total_tokens = plan->total_tokens;
    out->old_live_blocks = plan->old_live_blocks;
    out->new_live_blocks = plan->new_live_blocks;
    return REMP_OK;
}

remp_status remp_kv_plan_get_pair(const remp_kv_plan_t* plan, int32_t index, remp_kv_pair* out) {
    clear_error();
    if (!plan || !out) return fail(REMP_E_INVALID, "plan or out is NULL");
    if (index < 0 || index >= static_cast<int32_t>(plan->pairs.size()))
        return fail(REMP_E_RANGE, "pair index out of range");
    const Pair& p = plan->pairs[index];
    out->src = p.src;
    out->dst = p.dst;
    out->layer_begin = p.layer_begin;
    out->layer_end = p.layer_end;
    out->head_begin = p.head_begin;
    out->head_count = p.head_count;
    out->slice_bytes = p.slice_bytes;
    out->staging_bytes = p.slice_bytes * (p.layer_end - p.layer_begin);
    return REMP_OK;
}

remp_status remp_kv_plan_query(const remp_kv_plan_t* plan, int32_t src, int32_t dst, int64_t* staging_bytes,
                               int64_t* layer_offsets) {
    clear_error();
    if (!plan) return fail(REMP_E_INVALID, "plan is NULL");
    if (src < 0 || src >= plan->own_old.world()) return fail(REMP_E_RANGE, "src rank out of range");
    if (dst < 0 || dst >= plan->own_new.world()) return fail(REMP_E_RANGE, "dst rank out of range");
    const Pair* p = find_pair(*plan, src, dst);
    if (staging_bytes) *staging_bytes = p ? p->slice_bytes * (p->layer_end - p->layer_begin) : 0;
    if (layer_offsets) {
        for (int32_t l = 0; l <= plan->shape.num_layers; ++l) {
            if (!p) {
                layer_offsets[l] = 0;
                continue;
            }
            int32_t c = std::min(std::max(l, p->layer_begin), p->layer_end);
            layer_offsets[l] = static_cast<int64_t>(c - p->layer_begin) * p->slice_bytes;
        }
    }
    return REMP_OK;
}

remp_status remp_kv_workspace_bytes(const remp_kv_plan_t* plan, int64_t* bytes) {
    clear_error();
    if (!plan || !bytes) return fail(REMP_E_INVALID, "plan or bytes is NULL");
    *bytes = workspace_bytes(*plan);
    return REMP_OK;
}

const char* remp_status_string(remp_status st) {
    switch (st) {
        case REMP_OK: return "REMP_OK";
        case REMP_E_INVALID: return "REMP_E_INVALID";
        case REMP_E_UNSUPPORTED: return "REMP_E_UNSUPPORTED";
        case REMP_E_RANGE: return "REMP_E_RANGE";
        case REMP_E_CAPACITY: return "REMP_E_CAPACITY";
        case REMP_E_ALIGN: return "REMP_E_ALIGN";
        case REMP_E_SIZE: return "REMP_E_SIZE";
        case REMP_E_HIP: return "REMP_E_HIP";
    }
    return "REMP_E_UNKNOWN";
}

const char* remp_last_error(void) { return g_last_error.c_str(); }

const char* remp_kv_version(void) { return "0.1.0"; }

}  // extern "C"
