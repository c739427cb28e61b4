/*
 * A plain C99 program that runs a whole staged KV migration through the
 * library's C ABI (include/remp_kv.h) on the GPU, with device memory from
 * hipMalloc and a HIP stream of its own: no Python, no torch.
 *
 * Usage: gpu_consumer DIR
 * DIR holds the inputs the test wrote:
 *   meta.txt      L H D elem_bytes old_bs new_bs old_tp old_pp new_tp new_pp S old_nb new_nb old_nnz new_nnz
 *   tables.i32    seq_lens[S], old row_offsets[S+1], old ids[old_nnz], new row_offsets[S+1], new ids[new_nnz]
 *   old_R_L.bin   old rank R's layer L: K then V, [old_nb][old_bs][H_loc][D] elements each
 *   new_Q_L.bin   new rank Q's layer L before the migration (pre-fill), K then V
 * and receives:
 *   out_new_Q_L.bin   new rank Q's layer L after the migration
 *   out_st_R_Q.bin    the staging buffer of pair (R, Q)
 * Every old rank packs and every new rank unpacks, in two layer windows; only
 * the first pack and the first unpack expand the block tables, the other
 * calls reuse the descriptors (REMP_KV_REUSE_DESCRIPTORS).  Exits non-zero on
 * any failure, after printing it.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "remp_kv.h"

#define FAIL(...)                                  \
    do {                                           \
        fprintf(stderr, __VA_ARGS__);              \
        fprintf(stderr, "\n");                     \
        exit(1);                                   \
    } while (0)
#define HIP(call)                                                                          \
    do {                                                                                   \
        hipError_t e_ = (call);                                                            \
        if (e_ != hipSuccess) FAIL("%s: %s", #call, hipGetErrorString(e_));                \
    } while (0)
#define REMP(call)                                                                         \
    do {                                                                                   \
        remp_status s_ = (call);                                                           \
        if (s_ != REMP_OK) FAIL("%s: %s: %s", #call, remp_status_string(s_), remp_last_error()); \
    } while (0)

static const char* dir;

static void* read_file(const char* name, size_t expect) {
    char path[4096];
    snprintf(path, sizeof(path), "%s/%s", dir, name);
    FILE* f = fopen(path, "rb");
    if (!f) FAIL("cannot open %s", path);
    void* buf = malloc(expect ? expect : 1);
    if (!buf) FAIL("out of host memory");
    if (fread(buf, 1, expect, f) != expect) FAIL("%s is shorter than %zu bytes", path, expect);
    fclose(f);
    return buf;
}

static void write_file(const char* name, const void* data, size_t n) {
    char path[4096];
    snprintf(path, sizeof(path), "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f || fwrite(data, 1, n, f) != n) FAIL("cannot write %s", path);
    fclose(f);
}

/* first layer and layer count of a rank under equal contiguous ranges */
static void rank_layers(int32_t rank, int32_t tp, int32_t pp, int32_t L, int32_t* first, int32_t* count) {
    *count = L / pp;
    *first = (rank / tp) * *count;
}

static int32_t local_heads(int32_t H, int32_t tp) { return tp <= H ? H / tp : 1; }

int main(int argc, char** argv) {
    if (argc != 2) FAIL("usage: gpu_consumer DIR");
    dir = argv[1];
    char path[4096];
    snprintf(path, sizeof(path), "%s/meta.txt", dir);
    FILE* mf = fopen(path, "r");
    if (!mf) FAIL("cannot open %s", path);
    long long m[15];
    for (int i = 0; i < 15; ++i)
        if (fscanf(mf, "%lld", &m[i]) != 1) FAIL("meta.txt: value %d missing", i);
    fclose(mf);
    const int32_t L = (int32_t)m[0], H = (int32_t)m[1], D = (int32_t)m[2], eb = (int32_t)m[3];
    const int32_t bso = (int32_t)m[4], bsn = (int32_t)m[5];
    const int32_t tpo = (int32_t)m[6], ppo = (int32_t)m[7], tpn = (int32_t)m[8], ppn = (int32_t)m[9];
    const int32_t S = (int32_t)m[10];
    const int64_t nbo = m[11], nbn = m[12], nnzo = m[13], nnzn = m[14];

    const size_t nt = (size_t)S + 2 * ((size_t)S + 1) + (size_t)nnzo + (size_t)nnzn;
    int32_t* tab = (int32_t*)read_file("tables.i32", nt * 4);
    int32_t* lens = tab;
    int32_t* ooff = lens + S;
    int32_t* oids = ooff + S + 1;
    int32_t* noff = oids + nnzo;
    int32_t* nids = noff + S + 1;
    remp_block_tables old_tables = {S, lens, ooff, oids, nbo};
    remp_block_tables new_tables = {S, lens, noff, nids, nbn};

    remp_topo old_t = {tpo, ppo, NULL}, new_t = {tpn, ppn, NULL};
    remp_kv_shape shape = {L, H, D, eb, bso, bsn};
    remp_kv_plan_t* plan = NULL;
    REMP(remp_kv_plan(&old_t, &new_t, &shape, &old_tables, &plan));
    remp_kv_plan_info info;
    REMP(remp_kv_plan_get_info(plan, &info));
    const int32_t Wo = info.old_world, Wn = info.new_world;

    /* device tables */
    int32_t *d_lens, *d_ooff, *d_oids, *d_noff, *d_nids;
    HIP(hipMalloc((void**)&d_lens, (size_t)S * 4 + 4));
    HIP(hipMalloc((void**)&d_ooff, ((size_t)S + 1) * 4));
    HIP(hipMalloc((void**)&d_oids, (size_t)nnzo * 4 + 4));
    HIP(hipMalloc((void**)&d_noff, ((size_t)S + 1) * 4));
    HIP(hipMalloc((void**)&d_nids, (size_t)nnzn * 4 + 4));
    HIP(hipMemcpy(d_lens, lens, (size_t)S * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_ooff, ooff, ((size_t)S + 1) * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_oids, oids, (size_t)nnzo * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_noff, noff, ((size_t)S + 1) * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_nids, nids, (size_t)nnzn * 4, hipMemcpyHostToDevice));
    remp_dev_tables dev_old = {d_lens, d_ooff, d_oids};
    remp_dev_tables dev_new = {d_lens, d_noff, d_nids};

    /* pools: one allocation per (rank, layer), K then V */
    const size_t old_kv = (size_t)nbo * bso * local_heads(H, tpo) * D * eb;
    const size_t new_kv = (size_t)nbn * bsn * local_heads(H, tpn) * D * eb;
    void** old_mem = (void**)calloc((size_t)Wo * L, sizeof(void*));
    void** new_mem = (void**)calloc((size_t)Wn * L, sizeof(void*));
    void** old_k = (void**)calloc((size_t)Wo * L, sizeof(void*));
    void** old_v = (void**)calloc((size_t)Wo * L, sizeof(void*));
    void** new_k = (void**)calloc((size_t)Wn * L, sizeof(void*));
    void** new_v = (void**)calloc((size_t)Wn * L, sizeof(void*));
    remp_kv_pool* old_pool = (remp_kv_pool*)calloc((size_t)Wo, sizeof(remp_kv_pool));
    remp_kv_pool* new_pool = (remp_kv_pool*)calloc((size_t)Wn, sizeof(remp_kv_pool));
    for (int32_t r = 0; r < Wo; ++r) {
        int32_t first, count;
        rank_layers(r, tpo, ppo, L, &first, &count);
        for (int32_t i = 0; i < count; ++i) {
            char name[256];
            snprintf(name, sizeof(name), "old_%d_%d.bin", r, first + i);
            void* host = read_file(name, 2 * old_kv);
            void** slot = &old_mem[(size_t)r * L + i];
            HIP(hipMalloc(slot, 2 * old_kv));
            HIP(hipMemcpy(*slot, host, 2 * old_kv, hipMemcpyHostToDevice));
            free(host);
            old_k[(size_t)r * L + i] = *slot;
            old_v[(size_t)r * L + i] = (char*)*slot + old_kv;
        }
        old_pool[r].num_layers = count;
        old_pool[r].layout = REMP_KV_LAYOUT_NHD;
        old_pool[r].k = &old_k[(size_t)r * L];
        old_pool[r].v = &old_v[(size_t)r * L];
        old_pool[r].num_blocks = nbo;
    }
    for (int32_t q = 0; q < Wn; ++q) {
        int32_t first, count;
        rank_layers(q, tpn, ppn, L, &first, &count);
        for (int32_t i = 0; i < count; ++i) {
            char name[256];
            snprintf(name, sizeof(name), "new_%d_%d.bin", q, first + i);
            void* host = read_file(name, 2 * new_kv);
            void** slot = &new_mem[(size_t)q * L + i];
            HIP(hipMalloc(slot, 2 * new_kv));
            HIP(hipMemcpy(*slot, host, 2 * new_kv, hipMemcpyHostToDevice));
            free(host);
            new_k[(size_t)q * L + i] = *slot;
            new_v[(size_t)q * L + i] = (char*)*slot + new_kv;
        }
        new_pool[q].num_layers = count;
        new_pool[q].layout = REMP_KV_LAYOUT_NHD;
        new_pool[q].k = &new_k[(size_t)q * L];
        new_pool[q].v = &new_v[(size_t)q * L];
        new_pool[q].num_blocks = nbn;
    }

    /* staging: one buffer per pair, with its per-layer offsets */
    void** stage = (void**)calloc((size_t)Wo * Wn, sizeof(void*));
    int64_t* stage_bytes = (int64_t*)calloc((size_t)Wo * Wn, sizeof(int64_t));
    int64_t* offs = (int64_t*)calloc((size_t)Wo * Wn * (L + 1), sizeof(int64_t));
    for (int32_t r = 0; r < Wo; ++r)
        for (int32_t q = 0; q < Wn; ++q) {
            const size_t pq = (size_t)r * Wn + q;
            REMP(remp_kv_plan_query(plan, r, q, &stage_bytes[pq], &offs[pq * (L + 1)]));
            if (stage_bytes[pq] > 0) {
                HIP(hipMalloc(&stage[pq], (size_t)stage_bytes[pq]));
                HIP(hipMemset(stage[pq], 0xEE, (size_t)stage_bytes[pq]));
            }
        }

    int64_t ws_bytes = 0;
    REMP(remp_kv_workspace_bytes(plan, &ws_bytes));
    void* ws;
    HIP(hipMalloc(&ws, (size_t)ws_bytes));
    HIP(hipMemset(ws, 0, (size_t)ws_bytes));
    hipStream_t stream;
    HIP(hipStreamCreate(&stream));

    /* two layer windows; the first pack and the first unpack expand the tables */
    const int32_t cut = L / 2 > 0 ? L / 2 : L;
    const int32_t win[3] = {0, cut, L};
    int packed = 0, unpacked = 0;
    remp_buffer* out = (remp_buffer*)calloc((size_t)(Wn > Wo ? Wn : Wo), sizeof(remp_buffer));
    for (int w = 0; w < 2; ++w) {
        const int32_t l0 = win[w], l1 = win[w + 1];
        if (l0 == l1) continue;
        for (int32_t r = 0; r < Wo; ++r) {
            for (int32_t q = 0; q < Wn; ++q) {
                const size_t pq = (size_t)r * Wn + q;
                const int64_t a = offs[pq * (L + 1) + l0], z = offs[pq * (L + 1) + l1];
                out[q].ptr = (stage[pq] && z > a) ? (char*)stage[pq] + a : NULL;
                out[q].bytes = z - a;
            }
            REMP(remp_kv_pack(plan, r, l0, l1, &old_pool[r], &dev_old, out, ws, ws_bytes,
                              packed++ ? REMP_KV_REUSE_DESCRIPTORS : 0u, stream));
        }
        for (int32_t q = 0; q < Wn; ++q) {
            for (int32_t r = 0; r < Wo; ++r) {
                const size_t pq = (size_t)r * Wn + q;
                const int64_t a = offs[pq * (L + 1) + l0], z = offs[pq * (L + 1) + l1];
                out[r].ptr = (stage[pq] && z > a) ? (char*)stage[pq] + a : NULL;
                out[r].bytes = z - a;
            }
            REMP(remp_kv_unpack(plan, q, l0, l1, out, &new_pool[q], &new_tables, &dev_new, ws, ws_bytes,
                                unpacked++ ? REMP_KV_REUSE_DESCRIPTORS : 0u, stream));
        }
    }
    HIP(hipStreamSynchronize(stream));
    int32_t flag = -1;
    HIP(hipMemcpy(&flag, ws, 4, hipMemcpyDeviceToHost));
    printf("workspace flag %d\n", flag);
    if (flag != 0) FAIL("workspace flag %d after the migration", flag);

    /* the allocation-free unpack, whole cache in one call per new rank, into fresh copies of the new pools
       (the same starting bytes): every byte equal to what remp_kv_unpack wrote above */
    int noalloc_ranks = 0;
    if (ws_bytes <= REMP_KV_NOALLOC_SCRATCH_BYTES) {
        int32_t* d_status;
        HIP(hipMalloc((void**)&d_status, 4));
        HIP(hipMemset(d_status, 0x7F, 4));
        for (int32_t q = 0; q < Wn; ++q) {
            int32_t first, count;
            rank_layers(q, tpn, ppn, L, &first, &count);
            if (count == 0) continue;
            void** mem2 = (void**)calloc((size_t)count, sizeof(void*));
            void** k2 = (void**)calloc((size_t)count, sizeof(void*));
            void** v2 = (void**)calloc((size_t)count, sizeof(void*));
            for (int32_t i = 0; i < count; ++i) {
                char name[256];
                snprintf(name, sizeof(name), "new_%d_%d.bin", q, first + i);
                void* host = read_file(name, 2 * new_kv);
                HIP(hipMalloc(&mem2[i], 2 * new_kv));
                HIP(hipMemcpy(mem2[i], host, 2 * new_kv, hipMemcpyHostToDevice));
                free(host);
                k2[i] = mem2[i];
                v2[i] = (char*)mem2[i] + new_kv;
            }
            remp_kv_pool pool2 = new_pool[q];
            pool2.k = k2;
            pool2.v = v2;
            for (int32_t r = 0; r < Wo; ++r) {
                const size_t pq = (size_t)r * Wn + q;
                out[r].ptr = stage[pq];
                out[r].bytes = stage[pq] ? stage_bytes[pq] : 0;
            }
            REMP(remp_kv_unpack_noalloc(plan, q, 0, L, out, &pool2, &new_tables, &dev_new, d_status, 0u, stream));
            HIP(hipStreamSynchronize(stream));
            int32_t status = -1;
            HIP(hipMemcpy(&status, d_status, 4, hipMemcpyDeviceToHost));
            if (status != 0) FAIL("no-alloc unpack of rank %d: status %d", q, status);
            void* a_host = malloc(2 * new_kv);
            void* b_host = malloc(2 * new_kv);
            if (!a_host || !b_host) FAIL("out of host memory");
            for (int32_t i = 0; i < count; ++i) {
                HIP(hipMemcpy(a_host, new_mem[(size_t)q * L + i], 2 * new_kv, hipMemcpyDeviceToHost));
                HIP(hipMemcpy(b_host, mem2[i], 2 * new_kv, hipMemcpyDeviceToHost));
                if (memcmp(a_host, b_host, 2 * new_kv) != 0)
                    FAIL("no-alloc unpack of rank %d, layer %d differs from remp_kv_unpack", q, first + i);
                HIP(hipFree(mem2[i]));
            }
            free(a_host), free(b_host), free(mem2), free(k2), free(v2);
            ++noalloc_ranks;
        }
        HIP(hipFree(d_status));
    }
    printf("no-alloc unpack equal to remp_kv_unpack on %d ranks\n", noalloc_ranks);

    /* results */
    for (int32_t q = 0; q < Wn; ++q) {
        int32_t first, count;
        rank_layers(q, tpn, ppn, L, &first, &count);
        for (int32_t i = 0; i < count; ++i) {
            void* host = malloc(2 * new_kv);
            HIP(hipMemcpy(host, new_mem[(size_t)q * L + i], 2 * new_kv, hipMemcpyDeviceToHost));
            char name[256];
            snprintf(name, sizeof(name), "out_new_%d_%d.bin", q, first + i);
            write_file(name, host, 2 * new_kv);
            free(host);
        }
    }
    for (int32_t r = 0; r < Wo; ++r)
        for (int32_t q = 0; q < Wn; ++q) {
            const size_t pq = (size_t)r * Wn + q;
            if (!stage[pq]) continue;
            void* host = malloc((size_t)stage_bytes[pq]);
            HIP(hipMemcpy(host, stage[pq], (size_t)stage_bytes[pq], hipMemcpyDeviceToHost));
            char name[256];
            snprintf(name, sizeof(name), "out_st_%d_%d.bin", r, q);
            write_file(name, host, (size_t)stage_bytes[pq]);
            free(host);
            HIP(hipFree(stage[pq]));
        }

    for (size_t i = 0; i < (size_t)Wo * L; ++i)
        if (old_mem[i]) HIP(hipFree(old_mem[i]));
    for (size_t i = 0; i < (size_t)Wn * L; ++i)
        if (new_mem[i]) HIP(hipFree(new_mem[i]));
    HIP(hipFree(ws));
    HIP(hipFree(d_lens));
    HIP(hipFree(d_ooff));
    HIP(hipFree(d_oids));
    HIP(hipFree(d_noff));
    HIP(hipFree(d_nids));
    HIP(hipStreamDestroy(stream));
    remp_kv_plan_destroy(plan);
    free(old_mem), free(new_mem), free(old_k), free(old_v), free(new_k), free(new_v);
    free(old_pool), free(new_pool), free(stage), free(stage_bytes), free(offs), free(out), free(tab);
    printf("migration done: %d packs, %d unpacks\n", packed, unpacked);
    return 0;
}
