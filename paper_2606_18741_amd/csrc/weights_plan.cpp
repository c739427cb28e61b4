// Host planner of the weight-shard rebuild (Section 3.3): which byte ranges of
// the full host copy of every tensor form each rank's GPU shard.
#include <cstring>
#include <new>
#include <string>

#include "plan.hpp"
#include "weights_plan.hpp"

namespace remp {

void w_unit_range(int32_t t, int32_t tp, int32_t units, int32_t* u0, int32_t* n) {
    if (tp <= units) {
        *n = units / tp;
        *u0 = t * *n;
    } else {
        // more tensor ranks than units: each unit is kept by tp / units consecutive ranks
        *n = 1;
        *u0 = t / (tp / units);
    }
}

bool w_holds(const remp_w_plan_t& p, int32_t stage, const WTensor& w) {
    if (w.layer == REMP_W_FIRST_STAGE) return stage == 0;
    if (w.layer == REMP_W_LAST_STAGE) return stage == p.pp - 1;
    return p.stage_of_layer[w.layer] == stage;
}

int64_t w_part_rows(const remp_w_plan_t& p, const WPart& part, int32_t t) {
    if (part.split != REMP_W_SPLIT_ROWS) return part.rows;
    int32_t u0, n;
    w_unit_range(t, p.tp, part.units, &u0, &n);
    return part.rows / part.units * n;
}

void w_segments(const remp_w_plan_t& p, int32_t rank, int32_t tensor, std::vector<WSeg>& out) {
    const WTensor& w = p.tensors[tensor];
    const int32_t t = rank % p.tp;
    if (!w_holds(p, rank / p.tp, w)) return;
    const int64_t e = p.elem_bytes;
    int64_t dst = 0;
    for (int32_t k = 0; k < w.num_parts; ++k) {
        const WPart& a = p.parts[w.first_part + k];
        const int64_t row_bytes = a.cols * e;
        int32_t u0 = 0, n = 1;
        if (a.split != REMP_W_REPLICATED) w_unit_range(t, p.tp, a.units, &u0, &n);
        WSeg s;
        s.part = w.first_part + k;
        s.pitch = row_bytes;
        s.dst_off = dst;
        if (a.split == REMP_W_SPLIT_COLS) {
            const int64_t cpu = a.cols / a.units;   // columns per unit
            s.src_off = u0 * cpu * e;
            s.width = n * cpu * e;
            s.rows = a.rows;
        } else {
            const int64_t rpu = a.split == REMP_W_SPLIT_ROWS ? a.rows / a.units : a.rows;
            s.src_off = a.split == REMP_W_SPLIT_ROWS ? u0 * rpu * row_bytes : 0;
            s.width = row_bytes;
            s.rows = a.split == REMP_W_SPLIT_ROWS ? n * rpu : a.rows;
        }
        out.push_back(s);
        dst += s.rows * s.width;
    }
}

}  // namespace remp

using namespace remp;

extern "C" {

remp_status remp_w_plan(const remp_topo* topo, int32_t num_layers, int32_t elem_bytes, const remp_w_tensor* tensors,
                        int32_t num_tensors, remp_w_plan_t** out) {
    clear_error();
    if (!out) return fail(REMP_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!topo) return fail(REMP_E_INVALID, "topology is NULL");
    if (num_layers < 1) return fail(REMP_E_INVALID, "num_layers must be positive");
    if (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4)
        return fail(REMP_E_INVALID, "elem_bytes must be 1, 2 or 4");
    if (topo->tp < 1 || topo->pp < 1) return fail(REMP_E_INVALID, "topology needs TP >= 1 and PP >= 1");
    if (topo->pp > num_layers) return fail(REMP_E_INVALID, "topology has more pipeline stages than layers");
    if (topo->layer_starts) {
        if (topo->layer_starts[0] != 0 || topo->layer_starts[topo->pp] != num_layers)
            return fail(REMP_E_INVALID, "layer_starts must run from 0 to num_layers");
        for (int32_t s = 0; s < topo->pp; ++s)
            if (topo->layer_starts[s + 1] <= topo->layer_starts[s])
                return fail(REMP_E_INVALID, "layer_starts must increase (every stage holds a layer)");
    } else if (num_layers % topo->pp != 0) {
        return fail(REMP_E_UNSUPPORTED, "PP=" + std::to_string(topo->pp) + " does not divide num_layers=" +
                                            std::to_string(num_layers) + " (give layer_starts for an uneven split)");
    }
    if (num_tensors < 0) return fail(REMP_E_INVALID, "num_tensors < 0");
    if (num_tensors > 0 && !tensors) return fail(REMP_E_INVALID, "tensors is NULL");

    remp_w_plan_t* p = new (std::nothrow) remp_w_plan_t();
    if (!p) return fail(REMP_E_INVALID, "out of host memory");
    p->tp = topo->tp;
    p->pp = topo->pp;
    p->num_layers = num_layers;
    p->elem_bytes = elem_bytes;
    p->starts.resize(p->pp + 1);
    for (int32_t s = 0; s <= p->pp; ++s)
        p->starts[s] = topo->layer_starts ? topo->layer_starts[s]
                                          : static_cast<int32_t>(static_cast<int64_t>(s) * num_layers / p->pp);
    p->stage_of_layer.assign(num_layers, 0);
    for (int32_t s = 0; s < p->pp; ++s)
        for (int32_t l = p->starts[s]; l < p->starts[s + 1]; ++l) p->stage_of_layer[l] = s;

    auto reject = [&](remp_status st, const std::string& msg) {
        delete p;
        return fail(st, msg);
    };
    for (int32_t i = 0; i < num_tensors; ++i) {
        const remp_w_tensor& w = tensors[i];
        const std::string where = "tensor " + std::to_string(i);
        if (w.layer != REMP_W_FIRST_STAGE && w.layer != REMP_W_LAST_STAGE && (w.layer < 0 || w.layer >= num_layers))
            return reject(REMP_E_RANGE, where + ": layer out of range");
        if (w.num_parts < 1 || !w.parts) return reject(REMP_E_INVALID, where + ": needs at least one part");
        WTensor wt;
        wt.layer = w.layer;
        wt.first_part = static_cast<int32_t>(p->parts.size());
        wt.num_parts = w.num_parts;
        wt.shard_cols = -1;
        for (int32_t k = 0; k < w.num_parts; ++k) {
            const remp_w_part& a = w.parts[k];
            const std::string at = where + " part " + std::to_string(k);
            if (!a.host) return reject(REMP_E_INVALID, at + ": host pointer is NULL");
            if (a.rows < 1 || a.cols < 1) return reject(REMP_E_INVALID, at + ": sizes must be positive");
            if (a.rows > (int64_t(1) << 40) / a.cols) return reject(REMP_E_UNSUPPORTED, at + ": more than 2^40 elements");
            if (a.split != REMP_W_REPLICATED && a.split != REMP_W_SPLIT_ROWS && a.split != REMP_W_SPLIT_COLS)
                return reject(REMP_E_INVALID, at + ": unknown split");
            int64_t shard_cols = a.cols;
            if (a.split != REMP_W_REPLICATED) {
                const int64_t dim = a.split == REMP_W_SPLIT_ROWS ? a.rows : a.cols;
                if (a.units < 1 || dim % a.units != 0)
                    return reject(REMP_E_INVALID, at + ": units must be positive and divide the split dimension");
                if (a.units % p->tp != 0 && p->tp % a.units != 0)
                    return reject(REMP_E_INVALID, at + ": TP=" + std::to_string(p->tp) +
                                                      " neither divides nor is a multiple of units=" +
                                                      std::to_string(a.units));
                if (a.split == REMP_W_SPLIT_COLS) {
                    int32_t u0, n;
                    w_unit_range(0, p->tp, a.units, &u0, &n);
                    shard_cols = a.cols / a.units * n;
                }
            }
            if (wt.shard_cols >= 0 && wt.shard_cols != shard_cols)
                return reject(REMP_E_INVALID, at + ": shard column count differs from the tensor's other parts");
            wt.shard_cols = shard_cols;
            p->parts.push_back(WPart{static_cast<const char*>(a.host), a.rows, a.cols, a.split, a.units});
        }
        p->tensors.push_back(wt);
    }
    *out = p;
    return REMP_OK;
}

void remp_w_plan_destroy(remp_w_plan_t* plan) { delete plan; }

remp_status remp_w_shard_shape(const remp_w_plan_t* plan, int32_t rank, int32_t tensor, int64_t* rows,
                               int64_t* cols) {
    clear_error();
    if (!plan || !rows || !cols) return fail(REMP_E_INVALID, "plan, rows or cols is NULL");
    if (rank < 0 || rank >= plan->tp * plan->pp) return fail(REMP_E_RANGE, "rank out of range");
    if (tensor < 0 || tensor >= static_cast<int32_t>(plan->tensors.size()))
        return fail(REMP_E_RANGE, "tensor index out of range");
    const WTensor& w = plan->tensors[tensor];
    *rows = 0;
    *cols = 0;
    if (!w_holds(*plan, rank / plan->tp, w)) return REMP_OK;
    int64_t r = 0;
    for (int32_t k = 0; k < w.num_parts; ++k) r += w_part_rows(*plan, plan->parts[w.first_part + k], rank % plan->tp);
    *rows = r;
    *cols = w.shard_cols;
    return REMP_OK;
}

remp_status remp_w_shard_bytes(const remp_w_plan_t* plan, int32_t rank, int32_t tensor_begin, int32_t tensor_end,
                               int64_t* bytes) {
    clear_error();
    if (!plan || !bytes) return fail(REMP_E_INVALID, "plan or bytes is NULL");
    if (rank < 0 || rank >= plan->tp * plan->pp) return fail(REMP_E_RANGE, "rank out of range");
    if (tensor_begin < 0 || tensor_end < tensor_begin || tensor_end > static_cast<int32_t>(plan->tensors.size()))
        return fail(REMP_E_RANGE, "tensor window out of range");
    int64_t total = 0;
    for (int32_t i = tensor_begin; i < tensor_end; ++i) {
        int64_t r, c;
        remp_w_shard_shape(plan, rank, i, &r, &c);
        total += r * c * plan->elem_bytes;
    }
    *bytes = total;
    return REMP_OK;
}

}  // extern "C"
