/* A plain C99 client of libtreekv.so: the header compiles as C and the host-only entry points
 * (block manager, search controller, errors) work without Python or a GPU.  Built and run by
 * tests/test_c_client.py; prints "ok" and exits 0 when every check holds. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "treekv.h"

#define CHECK(c)                                                              \
    do {                                                                      \
        if (!(c)) {                                                           \
            fprintf(stderr, "%s:%d: %s (%s)\n", __FILE__, __LINE__, #c, tkv_last_error()); \
            return 1;                                                         \
        }                                                                     \
    } while (0)

int main(void) {
    tkv_bm* bm = NULL;
    int32_t toks[40], child = -1, blk[4], nblk = 0, sib = -1, tab[8], ntab = 0, kvlen = 0, freed[8], nfreed = 0;
    uint8_t hit[4];
    int32_t i, rc = 0;
    for (i = 0; i < 40; ++i) toks[i] = 100 + i;
    CHECK(tkv_bm_create(16, 16, 8, &bm) == TKV_OK);
    /* a 40-token sealed root takes blocks 0, 1, 2 (the last one partial) */
    CHECK(tkv_bm_extend(bm, -1, toks, 40, 1, &child, blk, hit, 4, &nblk) == TKV_OK);
    CHECK(child == 0 && nblk == 3 && blk[0] == 0 && blk[2] == 2 && !hit[0]);
    /* the same 20 tokens twice under the root: the second extension reuses both blocks */
    CHECK(tkv_bm_extend(bm, 0, toks, 20, 1, &child, blk, hit, 4, &nblk) == TKV_OK && child == 1);
    CHECK(tkv_bm_extend(bm, 0, toks, 20, 1, &sib, blk, hit, 4, &nblk) == TKV_OK && sib == 2);
    CHECK(nblk == 2 && hit[0] == 1 && hit[1] == 1);
    CHECK(tkv_bm_table(bm, 2, tab, 8, &ntab, &kvlen) == TKV_OK && ntab == 5 && kvlen == 60);
    CHECK(tkv_prune(bm, 2, freed, 8, &nfreed) == TKV_OK && nfreed == 0);    /* all blocks still held */
    CHECK(tkv_prune(bm, 2, freed, 8, &nfreed) == TKV_ENOSEQ);
    CHECK(strlen(tkv_last_error()) > 0);
    CHECK(tkv_bm_extend(bm, 0, toks, 40, 1, &child, blk, hit, 2, &nblk) == TKV_ECAP && nblk == 3);
    tkv_bm_destroy(bm);

    /* early pruning, k = 1: of two scored roots the lower one is pruned */
    {
        tkv_search* s = NULL;
        int32_t first = -1, flush = 0, batch[4], nb = 0, pruned[4], np = 0, st = 0, par = 0, dep = 0;
        float sc = 0.f, scores[2] = {0.25f, 0.75f};
        CHECK(tkv_search_create(1, 16, 0, 6, &s) == TKV_OK);
        CHECK(tkv_search_expand(s, -1, 3, &first) == TKV_OK && first == 0);
        CHECK(tkv_search_complete(s, 0, 50, &flush) == TKV_OK && flush == 1);   /* threshold 0 */
        CHECK(tkv_search_complete(s, 1, 60, &flush) == TKV_OK);
        CHECK(tkv_search_flush(s, batch, 4, &nb) == TKV_OK && nb == 2 && batch[0] == 0 && batch[1] == 1);
        CHECK(tkv_search_score(s, 2, batch, scores) == TKV_OK);
        CHECK(tkv_search_pruned(s, pruned, 4, &np) == TKV_OK && np == 1 && pruned[0] == 0);
        CHECK(tkv_search_node(s, 1, &st, &par, &dep, &sc) == TKV_OK && st == TKV_CAND_VERIFIED && sc == 0.75f);
        CHECK(tkv_search_score(s, 1, batch, scores) == TKV_EINVAL);            /* already scored */
        tkv_search_destroy(s);
    }
    if (rc == 0) printf("ok\n");
    return rc;
}
