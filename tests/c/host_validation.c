/*
 * Host-side validation of every KV-migration entry point, from plain C99, for
 * the sanitizer build: planning over many table shapes, and pack / unpack /
 * local copy / allocation-free unpack calls that either fail validation or
 * cover an empty layer window (validated completely, nothing launched).  The
 * device addresses are stand-ins that the host code never dereferences; no
 * call here reaches the GPU.  Prints one line per check, exits non-zero on a
 * failure.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
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

/* a stand-in device address, 256-byte aligned, never dereferenced by host code */
static void* fake(uintptr_t i) { return (void*)(uintptr_t)(0x7f0000000000ull + i * 0x10000000ull); }

/* S sequences of the given lengths, block size bs, ids 0..n-1 in a shuffled order, pad junk ids per row */
typedef struct {
    int32_t S;
    int32_t* lens;
    int32_t* offs;
    int32_t* ids;
    int64_t nblocks;
    remp_block_tables t;
} tables_t;

static tables_t make_tables(int32_t S, const int32_t* lens, int32_t bs, int32_t pad, uint32_t seed) {
    tables_t r;
    int64_t need = 0, i;
    int32_t s;
    r.S = S;
    r.lens = (int32_t*)malloc(sizeof(int32_t) * (size_t)(S > 0 ? S : 1));
    r.offs = (int32_t*)malloc(sizeof(int32_t) * (size_t)(S + 1));
    for (s = 0; s < S; ++s) {
        r.lens[s] = lens[s];
        need += (lens[s] + bs - 1) / bs;
    }
    r.nblocks = need + 3;
    r.ids = (int32_t*)malloc(sizeof(int32_t) * (size_t)(need + (int64_t)S * pad + 1));
    {
        int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * (size_t)r.nblocks);
        int64_t k = 0;
        for (i = 0; i < r.nblocks; ++i) perm[i] = (int32_t)i;
        for (i = r.nblocks - 1; i > 0; --i) { /* xorshift shuffle */
            int32_t tmp;
            int64_t j;
            seed ^= seed << 13;
            seed ^= seed >> 17;
            seed ^= seed << 5;
            j = (int64_t)(seed % (uint32_t)(i + 1));
            tmp = perm[i];
            perm[i] = perm[j];
            perm[j] = tmp;
        }
        r.offs[0] = 0;
        for (s = 0; s < S; ++s) {
            int32_t nb = (lens[s] + bs - 1) / bs, j;
            for (j = 0; j < nb; ++j) r.ids[r.offs[s] + j] = perm[k++];
            for (j = 0; j < pad; ++j) r.ids[r.offs[s] + nb + j] = -1;
            r.offs[s + 1] = r.offs[s] + nb + pad;
        }
        free(perm);
    }
    r.t.num_seqs = S;
    r.t.seq_lens = r.lens;
    r.t.row_offsets = r.offs;
    r.t.block_ids = r.ids;
    r.t.num_blocks = r.nblocks;
    return r;
}

static void free_tables(tables_t* r) {
    free(r->lens);
    free(r->offs);
    free(r->ids);
}

static void plans(void) {
    int32_t lens[6] = {5, 17, 0, 33, 1, 64};
    tables_t t = make_tables(6, lens, 16, 2, 7u);
    remp_topo a = {2, 1, NULL}, b = {1, 2, NULL}, rep = {8, 1, NULL};
    int32_t starts[4] = {0, 1, 3, 5};
    remp_topo uneven = {1, 3, starts};
    remp_kv_shape sh = {4, 8, 64, 2, 16, 16};
    remp_kv_shape sh5 = {5, 4, 64, 2, 16, 16};
    remp_kv_plan_t* p = NULL;
    int32_t saved;

    CHECK(remp_kv_plan(&a, &b, &sh, &t.t, &p) == REMP_OK && p, "plan with padded rows and an empty sequence");
    remp_kv_plan_destroy(p);
    p = NULL;
    CHECK(remp_kv_plan(&rep, &b, &sh, &t.t, &p) == REMP_OK && p, "plan with replicated old heads (TP8, H8)");
    remp_kv_plan_destroy(p);
    p = NULL;
    CHECK(remp_kv_plan(&a, &uneven, &sh5, &t.t, &p) == REMP_OK && p, "plan with an uneven partition");
    remp_kv_plan_destroy(p);
    p = NULL;
    saved = t.lens[1];
    t.lens[1] = -1;
    CHECK(remp_kv_plan(&a, &b, &sh, &t.t, &p) != REMP_OK && !p, "negative length refused");
    t.lens[1] = saved;
    saved = t.ids[t.offs[3]];
    t.ids[t.offs[3]] = (int32_t)t.nblocks;
    CHECK(remp_kv_plan(&a, &b, &sh, &t.t, &p) == REMP_E_RANGE && !p, "old id out of range refused");
    t.ids[t.offs[3]] = saved;
    saved = t.offs[4];
    t.offs[4] = t.offs[3];
    CHECK(remp_kv_plan(&a, &b, &sh, &t.t, &p) != REMP_OK && !p, "short row refused");
    t.offs[4] = saved;
    {
        remp_topo bad = {3, 1, NULL};
        CHECK(remp_kv_plan(&bad, &b, &sh, &t.t, &p) == REMP_E_UNSUPPORTED && !p, "TP 3 with 8 heads refused");
    }
    {
        int32_t bad_starts[3] = {0, 3, 2};
        remp_topo bad = {1, 2, bad_starts};
        CHECK(remp_kv_plan(&a, &bad, &sh5, &t.t, &p) == REMP_E_INVALID && !p, "decreasing partition refused");
    }
    free_tables(&t);
}

static void calls(void) {
    int32_t lens[4] = {40, 3, 0, 90};
    tables_t o = make_tables(4, lens, 16, 1, 11u);
    tables_t n = make_tables(4, lens, 32, 0, 13u);
    remp_topo ot = {2, 1, NULL}, nt = {4, 2, NULL};
    remp_kv_shape sh = {4, 8, 64, 2, 16, 32};
    remp_kv_plan_t* p = NULL;
    remp_kv_plan_info info;
    int64_t ws_bytes = 0, st_bytes = 0;
    void* ks[4];
    void* vs[4];
    remp_buffer staging[8];
    remp_dev_tables dt = {fake(100), fake(101), fake(102)};
    remp_kv_pool src, dst;
    int i, saved;
    void* ws = fake(200);

    CHECK(remp_kv_plan(&ot, &nt, &sh, &o.t, &p) == REMP_OK, "plan TP2/PP1 -> TP4/PP2");
    remp_kv_plan_get_info(p, &info);
    remp_kv_workspace_bytes(p, &ws_bytes);
    for (i = 0; i < 4; ++i) {
        ks[i] = fake(10 + 2 * i);
        vs[i] = fake(11 + 2 * i);
    }
    src.num_layers = 4;
    src.layout = REMP_KV_LAYOUT_NHD;
    src.k = ks;
    src.v = vs;
    src.num_blocks = o.nblocks;
    dst.num_layers = 2;
    dst.layout = REMP_KV_LAYOUT_NHD;
    dst.k = ks;
    dst.v = vs;
    dst.num_blocks = n.nblocks;
    for (i = 0; i < 8; ++i) {
        remp_kv_plan_query(p, 0, i, &st_bytes, NULL);
        staging[i].ptr = st_bytes ? fake(300 + i) : NULL;
        staging[i].bytes = st_bytes;
    }

    /* empty windows: everything validated, nothing launched */
    CHECK(remp_kv_pack(p, 0, 2, 2, &src, &dt, staging, ws, ws_bytes, 0, NULL) == REMP_OK, "pack, empty window");
    CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_OK,
          "unpack, empty window");
    CHECK(remp_kv_copy_local(p, 0, 3, 3, &src, &dt, &dst, &n.t, &dt, ws, ws_bytes, REMP_KV_REUSE_DESCRIPTORS, NULL) ==
              REMP_OK,
          "local copy, empty window");

    /* refusals before anything is enqueued */
    CHECK(remp_kv_pack(p, 9, 0, 4, &src, &dt, staging, ws, ws_bytes, 0, NULL) == REMP_E_RANGE, "pack: old rank");
    CHECK(remp_kv_pack(p, 0, 3, 2, &src, &dt, staging, ws, ws_bytes, 0, NULL) == REMP_E_RANGE, "pack: window");
    CHECK(remp_kv_pack(p, 0, 0, 4, &src, &dt, staging, ws, ws_bytes - 1, 0, NULL) == REMP_E_SIZE,
          "pack: small workspace");
    CHECK(remp_kv_pack(p, 0, 0, 4, &src, &dt, staging, (char*)ws + 16, ws_bytes, 0, NULL) == REMP_E_ALIGN,
          "pack: misaligned workspace");
    CHECK(remp_kv_pack(p, 0, 0, 4, &src, &dt, staging, ws, ws_bytes, 8, NULL) == REMP_E_INVALID, "pack: flags");
    staging[1].bytes -= 2;
    CHECK(remp_kv_pack(p, 0, 0, 4, &src, &dt, staging, ws, ws_bytes, 0, NULL) == REMP_E_SIZE, "pack: small staging");
    staging[1].bytes += 2;
    src.layout = 7;
    CHECK(remp_kv_pack(p, 0, 0, 4, &src, &dt, staging, ws, ws_bytes, 0, NULL) == REMP_E_INVALID, "pack: layout");
    src.layout = REMP_KV_LAYOUT_NHD;
    src.num_blocks = o.nblocks - 1;
    CHECK(remp_kv_pack(p, 0, 0, 4, &src, &dt, staging, ws, ws_bytes, 0, NULL) == REMP_E_SIZE, "pack: small pool");
    src.num_blocks = o.nblocks;

    saved = n.ids[n.offs[3]];
    n.ids[n.offs[3]] = n.ids[n.offs[0]];
    CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_INVALID,
          "unpack: a new id used twice");
    n.ids[n.offs[3]] = -5;
    CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_RANGE,
          "unpack: a new id out of range");
    n.ids[n.offs[3]] = saved;
    n.lens[1] += 1;
    CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_INVALID,
          "unpack: other lengths than planned");
    n.lens[1] -= 1;
    n.t.num_blocks = info.new_live_blocks - 1;
    CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_CAPACITY,
          "unpack: capacity");
    n.t.num_blocks = n.nblocks;
    CHECK(remp_kv_unpack(p, 0, 0, 2, NULL, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_INVALID,
          "unpack: no staging array");
    dst.num_layers = 3;
    CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_INVALID,
          "unpack: pool layer count");
    dst.num_layers = 2;
    {
        remp_dev_tables nodt = {NULL, NULL, NULL};
        CHECK(remp_kv_unpack(p, 0, 1, 1, staging, &dst, &n.t, &nodt, ws, ws_bytes, 0, NULL) == REMP_E_INVALID,
              "unpack: device tables missing");
    }
    CHECK(remp_kv_copy_local(p, 5, 0, 4, &src, &dt, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_RANGE,
          "local copy: rank in one topology only");
    {
        void* ok_k[2] = {fake(40), fake(42)};
        void* ok_v[2] = {fake(41), fake(43)};
        void* over_k[2] = {(char*)ks[0] + 64, fake(42)}; /* layer 0's new K storage inside its old K */
        dst.k = over_k;
        dst.v = ok_v;
        CHECK(remp_kv_copy_local(p, 0, 0, 2, &src, &dt, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_E_INVALID,
              "local copy: overlapping pools");
        dst.k = ok_k;
        CHECK(remp_kv_copy_local(p, 0, 1, 1, &src, &dt, &dst, &n.t, &dt, ws, ws_bytes, 0, NULL) == REMP_OK,
              "local copy: separate pools, empty window");
        dst.k = ks;
        dst.v = vs;
    }
    CHECK(remp_kv_unpack_noalloc(p, 0, 0, 2, staging, &dst, &n.t, &dt, (int32_t*)((char*)fake(400) + 2), 0, NULL) ==
              REMP_E_ALIGN,
          "no-alloc unpack: misaligned status");
    CHECK(remp_kv_unpack_noalloc(p, 0, 0, 2, staging, &dst, &n.t, &dt, NULL, 4, NULL) == REMP_E_INVALID,
          "no-alloc unpack: flags");
    remp_kv_plan_destroy(p);
    free_tables(&o);
    free_tables(&n);
}

static void big_noalloc(void) {
    /* one sequence of 2^22 tokens in blocks of 16: the workspace exceeds the static scratch */
    int32_t len = 1 << 22;
    tables_t t = make_tables(1, &len, 16, 0, 3u);
    remp_topo one = {1, 1, NULL};
    remp_kv_shape sh = {1, 1, 8, 2, 16, 16};
    remp_kv_plan_t* p = NULL;
    remp_buffer st = {fake(1), 0};
    void* k[1] = {fake(2)};
    void* v[1] = {fake(3)};
    remp_kv_pool pool = {1, REMP_KV_LAYOUT_NHD, k, v, t.nblocks};
    remp_dev_tables dt = {fake(4), fake(5), fake(6)};
    int64_t ws = 0;
    CHECK(remp_kv_plan(&one, &one, &sh, &t.t, &p) == REMP_OK, "plan with 262144 live blocks");
    remp_kv_workspace_bytes(p, &ws);
    CHECK(ws > REMP_KV_NOALLOC_SCRATCH_BYTES, "its workspace exceeds the static scratch");
    CHECK(remp_kv_unpack_noalloc(p, 0, 0, 1, &st, &pool, &t.t, &dt, NULL, 0, NULL) == REMP_E_SIZE,
          "no-alloc unpack refuses it");
    remp_kv_plan_destroy(p);
    free_tables(&t);
}

static void weights(void) {
    static uint16_t q[8 * 3], norm[3];
    remp_w_part qp = {q, 8, 3, REMP_W_SPLIT_ROWS, 2};
    remp_w_part np_ = {norm, 1, 3, REMP_W_REPLICATED, 1};
    remp_w_tensor ts[2] = {{0, 1, &qp}, {0, 1, &np_}};
    remp_topo tp2 = {2, 1, NULL};
    remp_w_plan_t* wp = NULL;
    int64_t rows = 0, cols = 0;
    CHECK(remp_w_plan(&tp2, 1, 2, ts, 2, &wp) == REMP_OK, "weight plan");
    CHECK(remp_w_shard_shape(wp, 1, 0, &rows, &cols) == REMP_OK && rows == 4 && cols == 3, "weight shard shape");
    CHECK(remp_w_load(wp, 2, 0, 2, NULL, 0, 0, NULL) == REMP_E_RANGE, "weight load: rank");
    CHECK(remp_w_load(wp, 0, 0, 3, NULL, 0, 0, NULL) == REMP_E_RANGE, "weight load: tensor window");
    CHECK(remp_w_load(wp, 0, 0, 2, NULL, 0, 0, NULL) == REMP_E_INVALID, "weight load: no destinations");
    remp_w_plan_destroy(wp);
}

int main(void) {
    plans();
    calls();
    big_noalloc();
    weights();
    printf("%d failures\n", failures);
    return failures ? 1 : 0;
}
