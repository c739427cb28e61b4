/*
 * remp_kv.h -- two-dimensional KV-cache migration for MI355X (gfx950).
 *
 * When a serving instance changes its tensor-parallel (TP) or pipeline-parallel
 * (PP) degree, every live K/V element keeps its identity but changes owner:
 * element KV[l, b, h] held by rank(l, h, T_old) must end up on rank(l, h, T_new)
 * (ReMP, Section 3.4.1).  TP changes re-slice the KV-head axis, PP changes
 * re-assign the layer axis.  This library
 *
 *   1. builds the migration plan on the host: which (old rank, new rank) pairs
 *      exchange which (layer, head-range) slices (Section 3.4.2, Algorithm 1);
 *   2. packs, on the GPU, an old rank's live paged K/V rows into one contiguous
 *      staging buffer per destination rank;
 *   3. unpacks, on the GPU, the staging buffers a new rank receives into its
 *      paged pool under the new block tables (the new tables are the block
 *      remapping that Section 3.4.5 allows; the block size may change).
 *
 * The transfer of staging buffers between GPUs (Section 3.4.3) is the
 * caller's: on one GPU the buffers simply stay in that GPU's memory.
 *
 * Conventions (readings of points the paper leaves open):
 *   - ranks:  rank(pp, tp) = pp * TP + tp;
 *   - layers: stage p of PP holds layers [p*L/PP, (p+1)*L/PP) (L % PP == 0),
 *             or the explicit partition remp_topo.layer_starts;
 *   - heads:  with TP <= H (H % TP == 0) tensor rank t holds KV heads
 *             [t*H/TP, (t+1)*H/TP); with TP > H (TP % H == 0, GQA replication)
 *             it holds the single head t*H/TP, so each head has TP/H replicas;
 *             a replicated head is taken from the destination itself if it
 *             holds a replica, else from old replica (its index among the
 *             head's new holders) mod (number of old replicas);
 *   - paged storage, per local layer, K and V separately:
 *       [num_blocks][block_size][H/TP][head_dim] elements of elem_bytes bytes,
 *     row-major; token t of sequence s lives in block ids[row_offsets[s] + t / block_size],
 *     slot t % block_size; only tokens t < seq_lens[s] are live;
 *   - staging of a pair (old rank r, new rank q): the pair's slices in ascending
 *     layer order; one slice is
 *       [kv: K then V][token: all sequences in order, live tokens only][head of the overlap][head_dim]
 *     so a slice is 2 * T * head_count * head_dim * elem_bytes bytes, T = sum of seq_lens,
 *     and any layer window is one contiguous byte range of the buffer.
 *
 * Elements are copied as raw bytes: any 1-, 2- or 4-byte type (fp8, fp16, bf16,
 * fp32 ...) moves bit for bit, NaN payloads and signed zeros included.
 *
 * Threading: plan objects are immutable after creation and may be shared by
 * threads.  The last-error text is per thread.  Pack and unpack are
 * stream-ordered and asynchronous; a workspace must not be used by two calls
 * that can run concurrently (different streams).  A plan must outlive the
 * stream work its calls enqueued only for as long as the call itself runs:
 * everything the kernels need is passed by value at launch.
 */
#ifndef REMP_KV_H
#define REMP_KV_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REMP_API __attribute__((visibility("default")))

typedef enum {
    REMP_OK = 0,
    REMP_E_INVALID = -1,     /* malformed argument: null pointer, inconsistent tables, duplicate block id */
    REMP_E_UNSUPPORTED = -2, /* valid request this version does not handle: L % PP != 0 without an
                                explicit partition, or TP neither divides nor is a multiple of the
                                KV head count */
    REMP_E_RANGE = -3,       /* rank, layer window or block id out of range */
    REMP_E_CAPACITY = -4,    /* the new pool cannot hold the live cache (Section 3.4.5, capacity) */
    REMP_E_ALIGN = -5,       /* a device pointer is not aligned to the element size */
    REMP_E_SIZE = -6,        /* a workspace or staging buffer is smaller than required */
    REMP_E_HIP = -7          /* a HIP runtime call or kernel launch failed */
} remp_status;

/* A parallel topology T = (TP, PP) (Section 3.4.1).  layer_starts (host,
 * PP + 1 entries, may be NULL) gives an explicit pipeline partition: stage p
 * holds layers [layer_starts[p], layer_starts[p+1]), starting at 0, ending at
 * num_layers, every stage holding at least one layer.  NULL means equal
 * contiguous ranges and then requires num_layers % PP == 0.  The plan copies
 * the array. */
typedef struct {
    int32_t tp;
    int32_t pp;
    const int32_t* layer_starts;
} remp_topo;

/* Model KV shape.  elem_bytes in {1, 2, 4}.  The block size may differ between
 * the old and the new pool. */
typedef struct {
    int32_t num_layers;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t elem_bytes;
    int32_t old_block_size;
    int32_t new_block_size;
} remp_kv_shape;

/* Block tables in host memory, CSR form: the row of sequence s is
 * block_ids[row_offsets[s] .. row_offsets[s+1]); only its first
 * ceil(seq_lens[s] / block_size) entries are read (the rest may be padding).
 * num_blocks is the capacity of the pool the ids index. */
typedef struct {
    int32_t num_seqs;
    const int32_t* seq_lens;     /* [num_seqs], >= 0 */
    const int32_t* row_offsets;  /* [num_seqs + 1], non-decreasing, row_offsets[0] >= 0 */
    const int32_t* block_ids;    /* [row_offsets[num_seqs]] */
    int64_t num_blocks;
} remp_block_tables;

/* The same three arrays in device memory (the GPU copy a serving engine keeps
 * for its attention kernels).  The contents must equal the host tables given
 * for the same role.  The kernels bound every access by the host sizes, so a
 * mismatch cannot make them read or write outside their buffers.  Device
 * tables that would index out of range (a negative length, a row or block id
 * outside the host sizes, more tokens than planned, a token with no old
 * source) are reported through the workspace flag (see
 * remp_kv_workspace_bytes); device tables that stay in range but differ from
 * the host tables are not detected, and then move other rows. */
typedef struct {
    const int32_t* seq_lens;
    const int32_t* row_offsets;
    const int32_t* block_ids;
} remp_dev_tables;

/* Physical layouts of a layer's K and V storage (H_loc = heads the rank holds). */
enum {
    REMP_KV_LAYOUT_NHD = 0,        /* K and V [num_blocks][block_size][H_loc][head_dim] */
    REMP_KV_LAYOUT_HND = 1,        /* K and V [num_blocks][H_loc][block_size][head_dim] */
    REMP_KV_LAYOUT_ROCM_SPLIT = 2  /* K [num_blocks][H_loc][head_dim/x][block_size][x], x = 16 / elem_bytes;
                                      V [num_blocks][H_loc][head_dim][block_size]
                                      (the ROCm paged-attention cache layout) */
};

/* A rank's paged KV storage: one K and one V device pointer per local layer
 * (local layer i = global layer first_layer_of_rank + i), each addressing
 * num_blocks blocks in `layout`.  Pointer arrays are host memory; entries for
 * layers outside the call's layer window may be NULL.  HND and ROCM_SPLIT need
 * head_dim * elem_bytes % 16 == 0 and 16-byte aligned storage; ROCM_SPLIT also
 * block_size * elem_bytes % 16 == 0 (REMP_E_UNSUPPORTED / REMP_E_ALIGN).  One
 * (block, head) tile of such a pool must fit the copy kernels' LDS budget:
 * block_size * (head_dim * elem_bytes + 16) <= 32768 (REMP_E_UNSUPPORTED). */
typedef struct {
    int32_t num_layers;
    int32_t layout;
    void* const* k;
    void* const* v;
    int64_t num_blocks;
} remp_kv_pool;

/* A device buffer and its size in bytes. */
typedef struct {
    void* ptr;
    int64_t bytes;
} remp_buffer;

/* Sizes of a plan. */
typedef struct {
    int32_t old_world;        /* TP_old * PP_old */
    int32_t new_world;        /* TP_new * PP_new */
    int32_t num_pairs;        /* (old rank, new rank) pairs that exchange data */
    int32_t num_items;        /* (old rank, new rank, layer) slices = Algorithm 1's send items */
    int64_t total_tokens;     /* T = sum of seq_lens */
    int64_t old_live_blocks;  /* sum of ceil(seq_lens / old_block_size) */
    int64_t new_live_blocks;  /* sum of ceil(seq_lens / new_block_size) */
} remp_kv_plan_info;

/* One pair: old rank src sends new rank dst the heads
 * [head_begin, head_begin + head_count) of layers [layer_begin, layer_end). */
typedef struct {
    int32_t src;
    int32_t dst;
    int32_t layer_begin;
    int32_t layer_end;
    int32_t head_begin;
    int32_t head_count;
    int64_t slice_bytes;      /* bytes of one layer's slice, K and V */
    int64_t staging_bytes;    /* (layer_end - layer_begin) * slice_bytes */
} remp_kv_pair;

typedef struct remp_kv_plan_s remp_kv_plan_t;

/* Flags of remp_kv_pack, remp_kv_unpack and remp_kv_copy_local. */
enum {
    /* Leave out the slices whose peer is the calling rank itself (the same
     * global rank id in the old and the new topology).  Those slices stay on
     * the worker (Section 3.4.3, local copy); move them with
     * remp_kv_copy_local instead of staging them.  Pack and unpack only. */
    REMP_KV_SKIP_LOCAL = 1u,
    /* Reuse the block descriptors an earlier call left in the workspace
     * instead of expanding the block tables again: the old ones (pack), the
     * new ones (unpack), or both (copy_local).  Meant for layer-wise streaming
     * (Section 3.4.4), where every window of a migration reads the same
     * tables: without it each call spends a few short kernels on the
     * expansion.  Every call that expands writes a stamp of the plan and the
     * tables it expanded into the workspace header; a reusing call's kernels
     * compare it with the stamp of their own plan and tables and, if it
     * differs (no earlier expansion, another plan, other new tables, or a
     * workspace overwritten since), copy nothing and set the workspace flag
     * to 2.  A reusing call leaves the flag otherwise as it was.  Host-side
     * validation is the same as without the flag. */
    REMP_KV_REUSE_DESCRIPTORS = 2u
};

/* Build the migration plan for T_old -> T_new (Section 3.4.2, Algorithm 1:
 * for every layer, intersect each new tensor rank's head range with each old
 * tensor rank's; every non-empty overlap is one send item of the old rank and
 * one receive item of the new rank, over all live blocks B).
 * Copies what it needs from old_tables; the caller may free them afterwards.
 * Validates shape (positive sizes, elem_bytes in {1,2,4}), divisibility
 * (REMP_E_UNSUPPORTED), table structure (REMP_E_INVALID) and old block ids in
 * [0, old_tables->num_blocks) (REMP_E_RANGE); at most 2^31 - 1 live tokens and
 * fewer than 2^28 live blocks in either block size (REMP_E_UNSUPPORTED).  On
 * failure *out is NULL.
 * Tuning hook (measurement only): if the environment variable
 * REMP_KV_WG_BYTES holds a positive integer when the plan is created, the copy
 * kernels launched with this plan aim to move about that many bytes per
 * workgroup instead of the built-in per-kernel targets (capped at 1 GiB).  It
 * changes launch shapes only, never the bytes written; later changes of the
 * environment do not affect an existing plan. */
REMP_API remp_status remp_kv_plan(const remp_topo* old_topo, const remp_topo* new_topo,
                         const remp_kv_shape* shape, const remp_block_tables* old_tables,
                         remp_kv_plan_t** out);

/* Free a plan; NULL is a no-op. */
REMP_API void remp_kv_plan_destroy(remp_kv_plan_t* plan);

REMP_API remp_status remp_kv_plan_get_info(const remp_kv_plan_t* plan, remp_kv_plan_info* out);

/* The i-th pair, pairs ordered by (src, dst); 0 <= index < num_pairs. */
REMP_API remp_status remp_kv_plan_get_pair(const remp_kv_plan_t* plan, int32_t index, remp_kv_pair* out);

/* Staging size of pair (src, dst) (0 if the pair exchanges nothing) and, if
 * layer_offsets is not NULL, its num_layers + 1 layer offsets: layer_offsets[l]
 * is the byte offset of the first slice of a layer >= l, so a window [l0, l1)
 * occupies bytes [layer_offsets[l0], layer_offsets[l1]). */
REMP_API remp_status remp_kv_plan_query(const remp_kv_plan_t* plan, int32_t src, int32_t dst,
                               int64_t* staging_bytes, int64_t* layer_offsets);

/* Workspace bytes needed by remp_kv_pack, remp_kv_unpack and
 * remp_kv_copy_local with this plan.  The workspace is device memory, 256-byte
 * aligned, owned by the caller; calls that share one must be ordered (one
 * stream).  After the stream work of a call that expands the tables completes,
 * its first 4 bytes (int32) hold 1 if the device tables would have made a
 * kernel index out of range (the cases listed at remp_dev_tables; those
 * accesses were skipped) and 0 otherwise; 2 means a call with
 * REMP_KV_REUSE_DESCRIPTORS found no matching descriptors and copied nothing.
 * Bytes 8-23 hold the stamps of the descriptors; the rest is scratch space of
 * the kernels. */
REMP_API remp_status remp_kv_workspace_bytes(const remp_kv_plan_t* plan, int64_t* bytes);

/* Pack (Section 3.4.2 send side, Section 3.4.3): for every slice old_rank sends
 * whose layer lies in [layer_begin, layer_end), copy its live rows from src
 * into the destination's staging buffer.  staging has new_world entries, by
 * destination rank; staging[q].ptr addresses the window's part of the (old_rank,
 * q) buffer, i.e. byte layer_offsets[layer_begin] of the whole buffer, and
 * staging[q].bytes must cover the window's slices.  Entries of ranks that get
 * nothing in the window may be {NULL, 0}.  Never writes src (the source
 * topology stays intact until the caller commits, Section 3.7).
 * old_tables: device copy of the tables given to remp_kv_plan.
 * flags: REMP_KV_SKIP_LOCAL (then staging[old_rank] is not used) and/or
 * REMP_KV_REUSE_DESCRIPTORS (old descriptors), or 0.
 * Everything is validated before anything is enqueued; on error nothing is. */
REMP_API remp_status remp_kv_pack(const remp_kv_plan_t* plan, int32_t old_rank,
                         int32_t layer_begin, int32_t layer_end,
                         const remp_kv_pool* src, const remp_dev_tables* old_tables,
                         const remp_buffer* staging,
                         void* workspace, int64_t workspace_bytes, uint32_t flags, hipStream_t stream);

/* Unpack (Section 3.4.2 receive side, Section 3.4.4 per layer window): for
 * every slice new_rank receives whose layer lies in [layer_begin, layer_end),
 * copy it from the source's staging buffer into dst at the live slots given by
 * new_tables.  staging has old_world entries, by source rank, addressed like
 * remp_kv_pack's.  Writes exactly the live (layer, token, head) rows of
 * new_rank's shard and nothing else.
 * new_tables (host) is validated: same sequences and lengths as the plan, rows
 * long enough, ids in [0, new_tables->num_blocks), no id used twice
 * (REMP_E_INVALID), enough blocks for the live cache (REMP_E_CAPACITY), and
 * dst->num_blocks >= new_tables->num_blocks (REMP_E_SIZE).
 * new_dev_tables: device copy of new_tables.
 * flags: REMP_KV_SKIP_LOCAL (then staging[new_rank] is not used) and/or
 * REMP_KV_REUSE_DESCRIPTORS (new descriptors; the new tables must be the ones
 * the descriptors were expanded from), or 0. */
REMP_API remp_status remp_kv_unpack(const remp_kv_plan_t* plan, int32_t new_rank,
                           int32_t layer_begin, int32_t layer_end,
                           const remp_buffer* staging,
                           const remp_kv_pool* dst, const remp_block_tables* new_tables,
                           const remp_dev_tables* new_dev_tables,
                           void* workspace, int64_t workspace_bytes, uint32_t flags, hipStream_t stream);

/* Allocation-free unpack, for callers that cannot allocate device memory or
 * pass a workspace: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid allocation.  Same arguments, validation and result as
 * remp_kv_unpack, but the workspace areas live in a static device array of the
 * library (8 MiB, REMP_KV_NOALLOC_SCRATCH_BYTES) instead of a caller buffer:
 * plans whose remp_kv_workspace_bytes exceeds that size are refused with
 * REMP_E_SIZE before anything is enqueued.  The call allocates no device
 * memory and calls no allocating routine; its first call on each device
 * resolves that device's copy of the array (hipGetSymbolAddress), so make it
 * outside graph capture; later calls only launch kernels.
 * status: NULL, or a 4-byte aligned device int32 that receives the status
 * flag remp_kv_workspace_bytes describes (0, 1 or 2); with NULL the flag stays
 * in the static array.
 * stream: NULL or a stream of the current device, whose copy of the array the
 * call uses; a stream of another device is refused (REMP_E_INVALID).
 * Every call on one device shares that device's array and finds the contents
 * the last call left: REMP_KV_REUSE_DESCRIPTORS reuses the descriptors of the
 * last expanding call on the device when their stamps match (flag 2
 * otherwise).  Calls that can overlap on one device (different streams, or
 * threads) race on the array and must be ordered by the caller. */
#define REMP_KV_NOALLOC_SCRATCH_BYTES (8 << 20)
REMP_API remp_status remp_kv_unpack_noalloc(const remp_kv_plan_t* plan, int32_t new_rank,
                                   int32_t layer_begin, int32_t layer_end,
                                   const remp_buffer* staging,
                                   const remp_kv_pool* dst, const remp_block_tables* new_tables,
                                   const remp_dev_tables* new_dev_tables,
                                   int32_t* status, uint32_t flags, hipStream_t stream);

/* Local copy (Section 3.4.3: when a slice's source and destination are the
 * same worker it is copied locally instead of transferred): for the slices
 * that `rank` sends to itself (same global rank id in both topologies) in
 * layers [layer_begin, layer_end), copy the live rows straight from src (the
 * rank's old pool, addressed by the planned old tables) into dst (its new
 * pool, addressed by new_tables), without staging.  Together with pack and
 * unpack called with REMP_KV_SKIP_LOCAL this yields the same new pool as a
 * staged migration while moving the local share once instead of twice.
 * rank must exist in both topologies.  The two pools may have any layouts
 * (HND or ROCM_SPLIT pools are copied in head tiles, through LDS when the two
 * layouts differ; those layouts need head_dim * elem_bytes % 16 == 0, a new
 * block size of at most 1024 and new_block_size * (head_dim * elem_bytes + 16)
 * <= 32768, REMP_E_UNSUPPORTED otherwise).  src and dst storage must not overlap
 * (checked per layer, REMP_E_INVALID).  new_tables are validated as in
 * remp_kv_unpack.  old_tables / new_dev_tables: device copies of the tables.
 * The workspace is the one remp_kv_workspace_bytes sizes; nothing is enqueued
 * on error.  flags: 0 or REMP_KV_REUSE_DESCRIPTORS (old and new descriptors). */
REMP_API remp_status remp_kv_copy_local(const remp_kv_plan_t* plan, int32_t rank,
                               int32_t layer_begin, int32_t layer_end,
                               const remp_kv_pool* src, const remp_dev_tables* old_tables,
                               const remp_kv_pool* dst, const remp_block_tables* new_tables,
                               const remp_dev_tables* new_dev_tables,
                               void* workspace, int64_t workspace_bytes, uint32_t flags, hipStream_t stream);

/* Measurement hook: while set (non-NULL), the calling thread's pack, unpack
 * and copy_local calls record `start` immediately before and `stop`
 * immediately after their copy kernel(s) on the call's stream.  Pass NULL,
 * NULL to clear. */
REMP_API void remp_kv_set_trace_events(hipEvent_t start, hipEvent_t stop);

REMP_API const char* remp_status_string(remp_status status);

/* Detail of the calling thread's last failure ("" if none). */
REMP_API const char* remp_last_error(void);

/* Library version, e.g. "0.1.0". */
REMP_API const char* remp_kv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* REMP_KV_H */
