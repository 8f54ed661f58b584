/*
 * A plain C99 consumer of the library: both public headers must compile as C
 * (gcc -std=c99 -pedantic -Werror) and the host-only entry points must work when
 * called from C through libkvx.so (no GPU needed): the work plan of a small batch,
 * argument errors with their messages, and a prefix-cache turn cycle.
 */
#include <stdio.h>
#include <string.h>

#include "kvx.h"
#include "kvx_cache.h"

#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            return 3;                                                      \
        }                                                                  \
    } while (0)

int main(void)
{
    /* two requests: P = 40, E = 100 and P = 0, E = 7; Hq 8 / Hkv 2, d 128 */
    int32_t prefix[2] = {40, 0}, extend[2] = {100, 7}, indptr[3] = {0, 9, 10};
    kvx_batch b;
    kvx_work_item items[64];
    int64_t count = -1, i;
    int64_t rows = 0;
    kvx_cache *cache = NULL;
    int32_t pre = -1, table[8], cached = -1;
    kvx_cache_counters st;

    b.num_reqs = 2;
    b.prefix_lens = prefix;
    b.extend_lens = extend;
    b.page_indptr = indptr;
    b.page_ids = NULL;
    CHECK(extend_attention_plan(&b, 8, 2, 128, 0, items, 64, &count) == KVX_OK);
    CHECK(count > 0 && count <= 64);
    for (i = 0; i < count; i++)
        if (items[i].req >= 0 && items[i].part < 0) rows += items[i].tok_count;
    CHECK(rows == 2 * (100 + 7)); /* every suffix token once per KV head */

    CHECK(extend_attention_plan(&b, 6, 4, 128, 0, NULL, 0, &count) == KVX_EINVAL);
    CHECK(strlen(kvx_last_error()) > 0);
    CHECK(extend_attention_plan(&b, 8, 2, 96, 0, NULL, 0, &count) == KVX_EUNSUPPORTED);

    CHECK(kvx_cache_create(16, 16, 64, KVX_EVICT_RR, &cache) == KVX_OK);
    CHECK(kvx_cache_begin_turn(cache, 7, 50, &pre, table, 8) == KVX_OK);
    CHECK(pre == 0);
    CHECK(kvx_cache_end_turn(cache, 7) == KVX_OK);
    CHECK(kvx_cache_agent(cache, 7, &cached, NULL, 0) == KVX_OK);
    CHECK(cached == 48); /* the prompt's three whole pages stay */
    CHECK(kvx_cache_begin_turn(cache, 7, 90, &pre, table, 8) == KVX_OK);
    CHECK(pre == 48);
    CHECK(kvx_cache_stats(cache, &st) == KVX_OK);
    CHECK(st.num_pages == 16 && st.active_agents == 1);
    CHECK(kvx_cache_destroy(cache) == KVX_OK);
    printf("C consumer: %lld plan items, cache cycle ok\n", (long long)count);
    return 0;
}
