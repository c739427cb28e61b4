/*
 * A plain C99 consumer of the library's C ABI (include/remp_kv.h, include/remp_weights.h),
 * exercising the host-only entry points: planning, sizing, queries, error reporting.
 * Prints one line per check and exits non-zero on the first failure.
 */
#include <stdio.h>
#include <string.h>

#include "remp_kv.h"
#include "remp_weights.h"

static int failures = 0;

#define CHECK(cond, what)                                                   \
    do {                                                                    \
        if (cond) {                                                         \
            printf("ok %s\n", what);                                        \
        } else {                                                            \
            printf("FAIL %s (%s)\n", what, remp_last_error());              \
            failures++;                                                     \
        }                                                                   \
    } while (0)

int main(void) {
    /* Two sequences of 5 and 17 tokens, block size 16: 1 + 2 live blocks. */
    int32_t lens[2] = {5, 17};
    int32_t offs[3] = {0, 1, 3};
    int32_t ids[3] = {3, 0, 2};
    remp_block_tables tables = {2, lens, offs, ids, 4};
    remp_topo old_t = {2, 1, NULL}, new_t = {1, 2, NULL};
    remp_kv_shape shape = {4, 8, 64, 2, 16, 16};
    remp_kv_plan_t* plan = NULL;

    CHECK(remp_kv_plan(&old_t, &new_t, &shape, &tables, &plan) == REMP_OK && plan != NULL, "plan TP2/PP1 -> TP1/PP2");

    remp_kv_plan_info info;
    memset(&info, 0, sizeof(info));
    CHECK(remp_kv_plan_get_info(plan, &info) == REMP_OK, "plan info");
    CHECK(info.total_tokens == 22 && info.old_live_blocks == 3 && info.new_live_blocks == 3, "token and block counts");

    /* old rank 0 holds heads 0-3 of every layer; new rank 0 holds layers 0-1, all heads:
       pair (0, 0) carries layers 0-1, heads 0-3: 2 layers * 2 (K, V) * 22 tokens * 4 heads * 64 * 2 bytes */
    int64_t bytes = -1, layer_offsets[5];
    CHECK(remp_kv_plan_query(plan, 0, 0, &bytes, layer_offsets) == REMP_OK, "query pair (0, 0)");
    CHECK(bytes == 2LL * 2 * 22 * 4 * 64 * 2, "staging bytes of pair (0, 0)");
    CHECK(layer_offsets[0] == 0 && layer_offsets[2] == bytes && layer_offsets[4] == bytes, "layer offsets");

    int64_t ws = 0;
    CHECK(remp_kv_workspace_bytes(plan, &ws) == REMP_OK && ws > 0 && ws % 256 == 0, "workspace size");

    remp_kv_plan_t* bad = NULL;
    remp_topo three = {3, 1, NULL};
    CHECK(remp_kv_plan(&three, &new_t, &shape, &tables, &bad) == REMP_E_UNSUPPORTED && bad == NULL,
          "TP that does not fit the head count is refused");
    CHECK(strlen(remp_last_error()) > 0, "last error text is set");
    CHECK(remp_kv_plan_query(plan, 9, 0, &bytes, NULL) == REMP_E_RANGE, "rank out of range");
    remp_kv_plan_destroy(plan);
    remp_kv_plan_destroy(NULL);

    /* weights: a 4-head Q projection [8][3] split by heads and a replicated norm [1][3], TP2 */
    static unsigned short q[8 * 3], norm[3];
    remp_w_part qp = {q, 8, 3, REMP_W_SPLIT_ROWS, 4};
    remp_w_part np = {norm, 1, 3, REMP_W_REPLICATED, 1};
    remp_w_tensor tensors[2] = {{0, 1, &qp}, {0, 1, &np}};
    remp_topo tp2 = {2, 1, NULL};
    remp_w_plan_t* wp = NULL;
    CHECK(remp_w_plan(&tp2, 1, 2, tensors, 2, &wp) == REMP_OK && wp != NULL, "weight plan TP2");
    int64_t rows = 0, cols = 0;
    CHECK(remp_w_shard_shape(wp, 1, 0, &rows, &cols) == REMP_OK && rows == 4 && cols == 3, "Q shard of rank 1");
    CHECK(remp_w_shard_shape(wp, 1, 1, &rows, &cols) == REMP_OK && rows == 1 && cols == 3, "norm shard");
    CHECK(remp_w_shard_bytes(wp, 0, 0, 2, &bytes) == REMP_OK && bytes == (4 * 3 + 3) * 2, "shard bytes");
    CHECK(remp_w_load(wp, 0, 0, 2, NULL, 0, 0, NULL) == REMP_E_INVALID, "load without destinations is refused");
    remp_w_plan_destroy(wp);

    CHECK(strcmp(remp_status_string(REMP_E_CAPACITY), "REMP_E_CAPACITY") == 0, "status names");
    printf("version %s\n", remp_kv_version());

    /* the headers' constants, for the binding to compare with */
#define CONST(name) printf("const %s %lld\n", #name, (long long)(name))
    CONST(REMP_OK);
    CONST(REMP_E_INVALID);
    CONST(REMP_E_UNSUPPORTED);
    CONST(REMP_E_RANGE);
    CONST(REMP_E_CAPACITY);
    CONST(REMP_E_ALIGN);
    CONST(REMP_E_SIZE);
    CONST(REMP_E_HIP);
    CONST(REMP_KV_SKIP_LOCAL);
    CONST(REMP_KV_REUSE_DESCRIPTORS);
    CONST(REMP_KV_LAYOUT_NHD);
    CONST(REMP_KV_LAYOUT_HND);
    CONST(REMP_KV_LAYOUT_ROCM_SPLIT);
    CONST(REMP_W_REPLICATED);
    CONST(REMP_W_SPLIT_ROWS);
    CONST(REMP_W_SPLIT_COLS);
    CONST(REMP_W_FIRST_STAGE);
    CONST(REMP_W_LAST_STAGE);
    CONST(REMP_W_COPY_ENGINE);
    return failures != 0;
}
