/*
 * The prefix store driven from plain C through include/ptstore.h: no Python,
 * no torch. Three objects are stored, their KV scattered from a paged cache,
 * then two requests are looked up and gathered into a second cache.
 * Expected values are fixed by hand (blocks of 2 tokens: A=(1,2) B=(3,4)
 * C=(5,6) D=(7,8)):
 *   insert  AB, ABC, ABD  -> ids A=0 B=1 C=2 D=3, 4 blocks stored
 *   lookup  ABD+CC        -> m=3, ids 0 1 3     (ABDC is not stored)
 *           BA            -> m=0                 (no root child B)
 * Every gathered byte must equal the byte scattered for that block. The
 * allocation-free lookup + gather must give the same m, ids and bytes.
 * A second store of 3 blocks refuses D: ptstore_insert_sync returns
 * PTSTORE_ERR_FULL with m = 2 3 2, then PTSTORE_OK for AB alone.
 * Exit status 0 and "abi_demo ok" on success.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ptstore.h"

#define CHECK(cond, msg)                                                          \
    do {                                                                          \
        if (!(cond)) {                                                            \
            fprintf(stderr, "abi_demo: %s (%s)\n", msg, ptstore_last_error());    \
            return 1;                                                             \
        }                                                                         \
    } while (0)

enum { L = 2, H = 1, D = 8, BT = 2, E = 2 };
enum { CHUNK = H * BT * D * E, BLOCK = L * 2 * CHUNK };

static int to_dev(void **d, const void *h, size_t n) {
    if (hipMalloc(d, n ? n : 16) != hipSuccess) return 1;
    return n && hipMemcpy(*d, h, n, hipMemcpyHostToDevice) != hipSuccess;
}

int main(void) {
    ptstore_config_t cfg = {.num_layers = L, .num_kv_heads = H, .head_dim = D, .block_tokens = BT,
                            .elem_bytes = E, .pool_blocks = 16, .index_slots = 0,
                            .hash_seed = 12345u, .flags = 0u, .host_blocks = 0, .replica_blocks = 0};
    ptstore_t *s = NULL;
    CHECK(ptstore_create(&cfg, &s) == PTSTORE_OK, "create");

    /* insert AB, ABC, ABD */
    const int32_t itok[] = {1, 2, 3, 4, 1, 2, 3, 4, 5, 6, 1, 2, 3, 4, 7, 8};
    const int64_t ioff[] = {0, 4, 10, 16};
    const int R = 3, MB = 3;
    void *dtok, *doff, *dm, *dids, *dcr, *dbt, *dcache;
    CHECK(!to_dev(&dtok, itok, sizeof itok) && !to_dev(&doff, ioff, sizeof ioff), "copy in");
    CHECK(hipMalloc(&dm, R * 4) == hipSuccess && hipMalloc(&dids, R * MB * 4) == hipSuccess &&
          hipMalloc(&dcr, R * MB) == hipSuccess, "alloc outputs");
    CHECK(ptstore_insert(s, dtok, doff, 16, R, MB, dm, dids, dcr, NULL) == PTSTORE_OK, "insert");

    /* the source cache holds R*MB blocks; block (r, b) sits at cache block r*MB+b */
    int32_t bt[9];
    for (int i = 0; i < R * MB; ++i) bt[i] = i;
    unsigned char *src = malloc((size_t)R * MB * BLOCK);
    for (size_t i = 0; i < (size_t)R * MB * BLOCK; ++i) src[i] = (unsigned char)(i * 131u + 7u);
    CHECK(!to_dev(&dbt, bt, sizeof bt) && !to_dev(&dcache, src, (size_t)R * MB * BLOCK), "cache in");
    CHECK(ptstore_scatter(s, dids, dcr, dbt, R, MB, dcache, R * MB, NULL) == PTSTORE_OK, "scatter");

    int32_t m[3], ids[9];
    uint8_t cr[9];
    CHECK(hipDeviceSynchronize() == hipSuccess, "sync");
    hipMemcpy(m, dm, sizeof m, hipMemcpyDeviceToHost);
    hipMemcpy(ids, dids, sizeof ids, hipMemcpyDeviceToHost);
    hipMemcpy(cr, dcr, sizeof cr, hipMemcpyDeviceToHost);
    const int32_t want_ids[9] = {0, 1, -1, 0, 1, 2, 0, 1, 3};
    const uint8_t want_cr[9] = {1, 1, 0, 0, 0, 1, 0, 0, 1};
    CHECK(m[0] == 2 && m[1] == 3 && m[2] == 3, "insert m");
    CHECK(!memcmp(ids, want_ids, sizeof ids) && !memcmp(cr, want_cr, sizeof cr), "insert ids");

    /* lookup + gather ABD+CC and BA into a 0xA5-filled cache */
    const int32_t qtok[] = {1, 2, 3, 4, 7, 8, 5, 6, 5, 6, 3, 4, 1, 2};
    const int64_t qoff[] = {0, 10, 14};
    const int QR = 2, QMB = 5;
    void *dq, *dqo, *dqm, *dqids, *dqbt, *dout;
    int32_t qbt[10];
    for (int i = 0; i < QR * QMB; ++i) qbt[i] = i;
    unsigned char *out = malloc((size_t)QR * QMB * BLOCK);
    memset(out, 0xA5, (size_t)QR * QMB * BLOCK);
    CHECK(!to_dev(&dq, qtok, sizeof qtok) && !to_dev(&dqo, qoff, sizeof qoff) &&
          !to_dev(&dqbt, qbt, sizeof qbt) && !to_dev(&dout, out, (size_t)QR * QMB * BLOCK), "q in");
    CHECK(hipMalloc(&dqm, QR * 4) == hipSuccess && hipMalloc(&dqids, QR * QMB * 4) == hipSuccess,
          "alloc q outputs");
    CHECK(ptstore_lookup_gather(s, dq, dqo, 14, QR, QMB, dqm, dqids, dqbt, dout, QR * QMB, NULL) ==
              PTSTORE_OK, "lookup_gather");
    CHECK(hipDeviceSynchronize() == hipSuccess, "sync 2");
    int32_t qm[2], qids[10];
    hipMemcpy(qm, dqm, sizeof qm, hipMemcpyDeviceToHost);
    hipMemcpy(qids, dqids, sizeof qids, hipMemcpyDeviceToHost);
    hipMemcpy(out, dout, (size_t)QR * QMB * BLOCK, hipMemcpyDeviceToHost);
    CHECK(qm[0] == 3 && qm[1] == 0, "lookup m");
    CHECK(qids[0] == 0 && qids[1] == 1 && qids[2] == 3 && qids[3] == -1 && qids[5] == -1, "lookup ids");

    /* gathered chunk (l, kv) of cache block b == scattered chunk of the block's creator */
    const int creator[4] = {0, 1, 5, 8}; /* source cache block of ids 0..3 */
    for (int b = 0; b < QR * QMB; ++b)
        for (int c = 0; c < 2 * L; ++c) {
            const unsigned char *got = out + ((size_t)c * QR * QMB + b) * CHUNK;
            if (b < 3) {
                const int id = qids[b];
                const unsigned char *exp = src + ((size_t)c * R * MB + creator[id]) * CHUNK;
                CHECK(!memcmp(got, exp, CHUNK), "gathered bytes");
            } else {
                for (int i = 0; i < CHUNK; ++i) CHECK(got[i] == 0xA5, "untouched bytes");
            }
        }
    /* the allocation-free call on the same inputs, into a second cache */
    void *dout2, *dqm2, *dqids2;
    unsigned char *fill = malloc((size_t)QR * QMB * BLOCK);
    memset(fill, 0xA5, (size_t)QR * QMB * BLOCK);
    CHECK(!to_dev(&dout2, fill, (size_t)QR * QMB * BLOCK), "noalloc cache in");
    CHECK(hipMalloc(&dqm2, QR * 4) == hipSuccess && hipMalloc(&dqids2, QR * QMB * 4) == hipSuccess,
          "alloc noalloc outputs");
    CHECK(ptstore_lookup_gather_noalloc(s, dq, dqo, 14, QR, QMB, dqm2, dqids2, dqbt, dout2, QR * QMB,
                                        NULL) == PTSTORE_OK, "lookup_gather_noalloc");
    CHECK(hipDeviceSynchronize() == hipSuccess, "sync 3");
    int32_t qm2[2], qids2[10];
    hipMemcpy(qm2, dqm2, sizeof qm2, hipMemcpyDeviceToHost);
    hipMemcpy(qids2, dqids2, sizeof qids2, hipMemcpyDeviceToHost);
    hipMemcpy(fill, dout2, (size_t)QR * QMB * BLOCK, hipMemcpyDeviceToHost);
    CHECK(!memcmp(qm, qm2, sizeof qm) && !memcmp(qids, qids2, sizeof qids) &&
          !memcmp(out, fill, (size_t)QR * QMB * BLOCK), "noalloc differs from lookup_gather");
    CHECK(ptstore_lookup_gather_noalloc(s, dq, dqo, 14, QR, PTSTORE_NOALLOC_MAX_ENTRIES, dqm2, dqids2,
                                        dqbt, dout2, QR * QMB, NULL) == PTSTORE_ERR_INVALID,
          "noalloc over its limit");

    ptstore_stats_t st;
    CHECK(ptstore_stats(s, &st) == PTSTORE_OK && st.blocks_stored == 4 && st.bad_entries == 0, "stats");
    CHECK(ptstore_destroy(s) == PTSTORE_OK, "destroy");

    /* a store of 3 blocks: D does not fit */
    cfg.pool_blocks = 3;
    CHECK(ptstore_create(&cfg, &s) == PTSTORE_OK, "create small");
    CHECK(ptstore_insert_sync(s, dtok, doff, 16, R, MB, dm, dids, dcr, NULL) == PTSTORE_ERR_FULL,
          "insert_sync on a full store");
    hipMemcpy(m, dm, sizeof m, hipMemcpyDeviceToHost);
    CHECK(m[0] == 2 && m[1] == 3 && m[2] == 2, "insert_sync m after the cut");
    CHECK(ptstore_insert_sync(s, dtok, doff, 4, 1, MB, dm, dids, dcr, NULL) == PTSTORE_OK,
          "insert_sync with nothing refused");
    CHECK(ptstore_stats(s, &st) == PTSTORE_OK && st.blocks_stored == 3 && st.full_events == 1,
          "stats of the small store");
    CHECK(ptstore_destroy(s) == PTSTORE_OK, "destroy small");
    printf("abi_demo ok\n");
    return 0;
}
