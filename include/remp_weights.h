/*
 * remp_weights.h -- GPU shard reconstruction from a host weight store, for MI355X (gfx950).
 *
 * ReMP keeps one full copy of the model's parameters in host memory shared by
 * the workers (Section 3.3).  On a topology switch every worker rebuilds its
 * GPU-resident shard for the target topology from that copy instead of
 * reloading checkpoints: the pipeline stage decides which layers' tensors a
 * worker keeps, the tensor rank decides which slice of each partitioned
 * tensor it keeps, and replicated tensors are kept whole (Section 3.3).  The
 * rebuild runs concurrently with the KV-cache migration, so the switch's
 * critical path is the slower of the two (Section 3.2).
 *
 * This library plans, for one target topology, which byte ranges of the
 * store form each shard, and copies them host -> HBM on a caller stream in one
 * pass (slicing and transfer together, no host-side repacking):
 *
 *   - by default with a gather kernel that reads the page-locked store over
 *     PCIe and writes the shard into HBM; its grid can be capped so that it
 *     leaves most compute units to a KV migration running beside it;
 *   - with REMP_W_COPY_ENGINE, with the GPU's DMA engines (one 2-D copy per
 *     part), which uses no compute units at all.
 *
 * Conventions (readings of points the paper leaves open; they are those of the
 * usual Megatron-style tensor parallelism):
 *   - ranks and layers as in remp_kv.h: rank(pp, tp) = pp * TP + tp, stage p
 *     holds layers [p*L/PP, (p+1)*L/PP) or the explicit remp_topo.layer_starts;
 *   - a store tensor is row-major [rows][cols] of elem_bytes-byte elements;
 *   - a partitioned tensor is split along one dimension into `units` equal
 *     units (attention heads, or single rows / columns); with TP <= units
 *     (units % TP == 0) tensor rank t keeps units [t*units/TP, (t+1)*units/TP);
 *     with TP > units (TP % units == 0, e.g. KV heads under GQA) it keeps the
 *     single unit t*units/TP, so each unit is replicated on TP/units ranks;
 *   - column-parallel projections (attention Q, K, V; MLP gate and up; vocab
 *     embedding and LM head) split their output rows, row-parallel ones
 *     (attention output, MLP down) their input columns;
 *   - a GPU tensor may stack several store tensors along rows (fused Q|K|V,
 *     fused gate|up): its shard is the rank's slice of each part, in order.
 *
 * Memory: the store must be page-locked host memory allocated with
 * hipHostMalloc (torch: pin_memory=True); load checks every source range and
 * refuses pageable memory, which the GPU cannot read.  Shard buffers are the
 * caller's device memory, each contiguous [shard rows][shard cols].
 *
 * Threading: a plan is immutable after creation and may be shared by threads.
 * Loads are stream-ordered and asynchronous; the store must stay allocated and
 * unchanged until the stream work completes.
 */
#ifndef REMP_WEIGHTS_H
#define REMP_WEIGHTS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "remp_kv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* How a store tensor is partitioned among tensor ranks. */
typedef enum {
    REMP_W_REPLICATED = 0,  /* every tensor rank keeps all of it (norm weights, biases) */
    REMP_W_SPLIT_ROWS = 1,  /* column-parallel: rows split into units */
    REMP_W_SPLIT_COLS = 2   /* row-parallel: columns split into units */
} remp_w_split;

/* Layer value of tensors outside the decoder layers. */
#define REMP_W_FIRST_STAGE (-1)  /* held by pipeline stage 0 (token embedding) */
#define REMP_W_LAST_STAGE (-2)   /* held by the last stage (final norm, LM head) */

/* One store tensor contributing to a GPU tensor. */
typedef struct {
    const void* host;   /* full tensor, row-major [rows][cols], page-locked host memory */
    int64_t rows;       /* >= 1 */
    int64_t cols;       /* >= 1 */
    int32_t split;      /* remp_w_split */
    int32_t units;      /* split granularity: the split dimension must be a multiple of it
                           (ignored when replicated) */
} remp_w_part;

/* One GPU tensor of the model: its parts stack along rows in the shard, and
 * every part must give the same shard column count. */
typedef struct {
    int32_t layer;             /* decoder layer in [0, num_layers), or REMP_W_FIRST_STAGE / REMP_W_LAST_STAGE */
    int32_t num_parts;         /* >= 1 */
    const remp_w_part* parts;  /* host array of num_parts entries */
} remp_w_tensor;

/* REMP_W_COPY_ENGINE: copy with the DMA engines instead of the gather kernel. */
#define REMP_W_COPY_ENGINE 1u

typedef struct remp_w_plan_s remp_w_plan_t;

/* Plan the shards of every rank of `topo` for a model of num_layers decoder
 * layers.  The plan copies the tensor and part descriptors (not the store's
 * bytes: it keeps the host pointers).  Host-only; checks the topology
 * (REMP_E_UNSUPPORTED for L % PP != 0 without a partition), layers
 * (REMP_E_RANGE), null pointers, non-positive sizes, units that do not divide
 * the split dimension, TP that neither divides nor is a multiple of a part's
 * units, and parts of one tensor with different shard column counts
 * (REMP_E_INVALID).  elem_bytes in {1, 2, 4}.  On failure *out is NULL. */
REMP_API remp_status remp_w_plan(const remp_topo* topo, int32_t num_layers, int32_t elem_bytes,
                                 const remp_w_tensor* tensors, int32_t num_tensors, remp_w_plan_t** out);

/* Free a plan; NULL is a no-op. */
REMP_API void remp_w_plan_destroy(remp_w_plan_t* plan);

/* Shard shape of `tensor` on `rank`, in elements; 0 x 0 when the rank's stage
 * does not hold the tensor.  REMP_E_RANGE for a bad rank or tensor index. */
REMP_API remp_status remp_w_shard_shape(const remp_w_plan_t* plan, int32_t rank, int32_t tensor,
                                        int64_t* rows, int64_t* cols);

/* Total shard bytes of `rank` over tensors [tensor_begin, tensor_end). */
REMP_API remp_status remp_w_shard_bytes(const remp_w_plan_t* plan, int32_t rank, int32_t tensor_begin,
                                        int32_t tensor_end, int64_t* bytes);

/* Build the shards of `rank` for tensors [tensor_begin, tensor_end) on `stream`.
 *
 * dst: host array indexed by tensor index (all num_tensors entries addressable);
 *      dst[i] for a tensor the rank holds, inside the window, is its device
 *      buffer of shard rows * cols * elem_bytes bytes; other entries are ignored
 *      and may be NULL.
 * max_workgroups: cap on the gather kernel's grid (0: the library's default);
 *      ignored with REMP_W_COPY_ENGINE.
 *
 * Before any copy is enqueued it checks that every source range lies in
 * page-locked host memory (REMP_E_INVALID otherwise), that every destination
 * is device memory with room for its shard (REMP_E_INVALID / REMP_E_SIZE), and
 * that destinations are aligned to elem_bytes (REMP_E_ALIGN).  On any error
 * nothing is enqueued.  Never writes the store. */
REMP_API remp_status remp_w_load(const remp_w_plan_t* plan, int32_t rank, int32_t tensor_begin, int32_t tensor_end,
                                 void* const* dst, uint32_t flags, int32_t max_workgroups, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* REMP_WEIGHTS_H */
