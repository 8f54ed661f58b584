/*
 * kvx_cache.h -- host-side prefix cache for multi-turn agents over the kvx page
 * pool: per-agent cached histories, page allocation, and eviction by round-robin
 * tail chunks (paper Section 3.2, Algorithm 1) or by least-recent leaf nodes (the
 * LRU baseline of Sections 3.1 and 4).
 *
 * The model.  Every agent (trajectory) owns a private cached history: the first
 * `cached` tokens of its context, held in whole pages of the pool (no sharing
 * between agents, as in the analysis of Section 3.3).  Each finished turn adds one
 * node to the agent's path: the full pages its prompt added to the cache.  A turn
 * start and a turn end both stamp every node of the agent's path with the current
 * logical time, so one agent's nodes always share one time stamp (the recency
 * synchronization of Section 3.1).  While a turn runs the agent is active and its
 * pages are pinned; between turns it is idle and its pages may be evicted.
 *
 * Eviction reclaims the pages a turn start needs beyond the free ones:
 *   KVX_EVICT_LRU  repeatedly drops the whole leaf node with the oldest time stamp
 *                  among idle agents (ties: smaller agent id); removing a leaf
 *                  exposes its parent.
 *   KVX_EVICT_RR   Algorithm 1: the idle agents holding pages form one queue in
 *                  agent-id order, starting after the agent that lost the last
 *                  chunk of any earlier reclamation (the round robin continues
 *                  across reclamations).  The front agent loses one tail chunk:
 *                  min(chunk, pages of its leaf node, pages still to reclaim)
 *                  pages from the end of its leaf; it goes to the back of the
 *                  queue while it holds pages.  Eligibility (idle, non-empty) is
 *                  rechecked at every pop.
 * Completion signals (Section 3.2, "Handling stale agent trajectories") are
 * kvx_cache_complete: the agent's pages are freed at once.  Without them, the
 * same passage's recency tiering keeps stale agents from holding pages for many
 * rounds: kvx_cache_set_recency_tiers.
 *
 * Host tier (optional; the paper's future work, Section 6: idle state spilled to
 * CPU memory and reloaded instead of recomputed).  A tiered cache also manages
 * `host_pages` page records of a caller-owned pinned host buffer (see
 * kv_pool_spill / kv_pool_reload in kvx.h).  An idle agent's history is then its
 * device pages followed, without a gap, by its host pages.  Pages the policy
 * evicts are spilled to host records instead of dropped, farthest page first; a
 * spill that finds every record taken first drops the oldest record whose owner
 * is idle (that owner's farthest host page), and if every record belongs to an
 * agent inside a turn the page is dropped instead.  A turn start reuses device
 * pages, then host pages, up to the prompt's limit; the reused host pages are
 * reloaded into freshly allocated device pages and their records freed, so an
 * agent inside a turn holds no host pages.
 *
 * Shared prefixes (Section 2: agents typically share a short common prefix such
 * as a system prompt, kept in the radix tree; eviction starts at idle leaves and
 * exposes parents, Section 3.1).  Agents that join a group share its first S
 * whole pages: one node, present or absent as a whole, that every member's page
 * table reads.  A member's history is the group node, then its private pages,
 * then its host pages; a member holds private pages only while the node is
 * present.  The first member turn that computes the span creates the node from
 * its own pages; copies computed concurrently by other members are freed at their
 * turn end.  The node is a leaf -- evictable, whole, never spilled -- only while
 * no member is inside a turn and no member holds private or host pages.  Its
 * stamp is the last turn start or end of any member: LRU weighs it among the
 * leaves by that stamp; round robin reclaims it after the agents' queue, oldest
 * first.
 *
 * Conventions: every call is synchronous host code, returns KVX_OK or a
 * kvx_status code from kvx.h (kvx_last_error() describes the failure), and is not
 * thread-safe for one cache (callers serialize calls on a cache).  Page ids are
 * indices into a kvx pool of the same num_pages; the cache never touches the pool's
 * memory.  A cache is owned by the library until kvx_cache_destroy.
 */
#ifndef KVX_CACHE_H
#define KVX_CACHE_H

#include <stdint.h>

#include "kvx.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kvx_cache kvx_cache; /* opaque; owned by the library */

enum kvx_evict_policy {
    KVX_EVICT_LRU = 0, /* whole least-recent leaf nodes */
    KVX_EVICT_RR = 1   /* round-robin tail chunks (Algorithm 1) */
};

typedef struct {
    int64_t num_pages;      /* pool pages managed */
    int64_t free_pages;     /* pages owned by nobody */
    int64_t cached_pages;   /* pages of idle and active agents' cached histories */
    int64_t turn_pages;     /* pages allocated to running turns beyond their cached prefix */
    int64_t evicted_pages;  /* pages reclaimed by eviction since creation */
    int64_t evictions;      /* eviction steps (LRU nodes or RR chunks) since creation */
    int32_t agents;         /* agents known to the cache */
    int32_t active_agents;  /* agents inside a turn */
    int64_t host_pages;     /* host records managed (0: no host tier) */
    int64_t host_used;      /* records holding a spilled page */
    int64_t spilled_pages;  /* pages spilled since creation */
    int64_t reloaded_pages; /* pages reloaded since creation */
    int64_t host_dropped_pages; /* records dropped to make room since creation */
    int64_t group_pages;    /* pages of present shared-prefix group nodes */
} kvx_cache_counters;

/* Page moves a tiered turn start asks for, to run on the pool in this order
 * before the turn's store_kv: first every spill (kv_pool_spill of
 * spill_pages[i] into record spill_slots[i]), then every reload (kv_pool_reload
 * of record reload_slots[i] into page reload_pages[i]).  Moves of successive
 * calls must run in call order (one stream). */
typedef struct {
    const int32_t *spill_pages;   /* [n_spill]; the four arrays are owned by the cache and */
    const int32_t *spill_slots;   /* stay valid until the next call on it                  */
    const int32_t *reload_pages;  /* [n_reload] */
    const int32_t *reload_slots;
    int64_t n_spill;
    int64_t n_reload;
} kvx_cache_moves;

/*
 * Create a cache over `num_pages` pages of `page_size` tokens.
 *   page_size     16 (the pool's page size).
 *   chunk_tokens  RR tail-chunk size in tokens, a positive multiple of page_size
 *                 (the paper evaluates 1024); ignored by LRU but still checked.
 *   policy        KVX_EVICT_LRU or KVX_EVICT_RR.
 * Errors: EINVAL (sizes, policy, out NULL), EUNSUPPORTED (page_size), ENOMEM.
 */
int kvx_cache_create(int64_t num_pages, int32_t page_size, int32_t chunk_tokens, int32_t policy,
                     kvx_cache **out);

/*
 * A cache with a host tier of `host_pages` >= 0 records (0: the same as
 * kvx_cache_create).  Record r is bytes [r * R, (r + 1) * R) of the caller's
 * pinned host buffer, R = kv_pool_record_bytes of the pool.  Turns of a cache
 * with host_pages > 0 start with kvx_cache_begin_turn_tiered.  Errors: as
 * kvx_cache_create, and EINVAL for host_pages outside [0, 2^31 - 1].
 */
int kvx_cache_create_tiered(int64_t num_pages, int64_t host_pages, int32_t page_size, int32_t chunk_tokens,
                            int32_t policy, kvx_cache **out);

/*
 * Recency tiering for KVX_EVICT_RR (Section 3.2, for stale trajectories when no
 * completion signal arrives; the paper does not evaluate it).  With
 * tier_width > 0, each reclamation groups the idle agents holding pages into
 * tiers by age = (logical clock - the agent's last stamp) / tier_width, where
 * the clock ticks once per turn start and once per turn end; it visits the
 * tiers from the oldest to the newest and runs the round robin within each,
 * moving on once a tier holds nothing evictable.  0 (the default) turns it off.
 * Errors: EINVAL (NULL cache, tier_width < 0, an LRU cache).
 */
int kvx_cache_set_recency_tiers(kvx_cache *cache, int64_t tier_width);

/* Free a cache.  NULL is a no-op. */
int kvx_cache_destroy(kvx_cache *cache);

/*
 * Start a turn of `agent` (any id; an unknown agent starts with nothing cached)
 * whose prompt is `prompt_len` >= 1 tokens: its context so far, then the new
 * input.  The reused prefix is the cached history capped at the last whole page
 * before the prompt's final token (a turn always computes at least one token):
 *   *prefix_len = min(cached, page_size * floor((prompt_len - 1) / page_size)).
 * Cached pages past *prefix_len are dropped.  The pages for tokens
 * [*prefix_len, prompt_len) are then allocated, evicting idle agents' pages per
 * the policy when too few are free.  On success page_ids[0 .. n) with
 * n = ceil(prompt_len / page_size) holds the turn's page table (logical page j ->
 * physical page), ready for store_kv / extend_attention with P = *prefix_len and
 * E = prompt_len - *prefix_len, and the agent is active.
 *   page_ids, cap  host buffer of cap >= n entries (checked before any change).
 * Errors: EINVAL (agent already active, prompt_len < 1, cap, NULL pointers),
 * ENOMEM (not enough pages even after evicting every idle page: the pages
 * evicted so far stay evicted, the agent stays idle with its prefix).
 */
int kvx_cache_begin_turn(kvx_cache *cache, int64_t agent, int32_t prompt_len, int32_t *prefix_len,
                         int32_t *page_ids, int64_t cap);

/*
 * kvx_cache_begin_turn on a cache of any kind, also returning the page moves it
 * needs (`moves`, filled on success and on ENOMEM; on ENOMEM only spills are
 * listed, and they must still run).  *prefix_len counts the reused device pages
 * and the reloaded host pages.  Errors: as kvx_cache_begin_turn, and EINVAL for
 * moves == NULL (checked first).  kvx_cache_begin_turn on a cache with a host
 * tier fails with EINVAL (its spills would be lost).
 */
int kvx_cache_begin_turn_tiered(kvx_cache *cache, int64_t agent, int32_t prompt_len, int32_t *prefix_len,
                                int32_t *page_ids, int64_t cap, kvx_cache_moves *moves);

/*
 * End the running turn of `agent`: the prompt's whole pages stay cached as the
 * agent's history (a new node holding the pages this turn added), its partial
 * last page is freed, and the agent becomes idle.  Errors: EINVAL (not active).
 */
int kvx_cache_end_turn(kvx_cache *cache, int64_t agent);

/*
 * Completion signal: free every page of an idle `agent` and forget it.
 * Errors: EINVAL (unknown or active agent).
 */
int kvx_cache_complete(kvx_cache *cache, int64_t agent);

/*
 * Private cached history of `agent` in tokens (0 for an unknown agent; a group's
 * shared pages are not counted, see kvx_cache_group) and, if `page_ids`
 * is non-NULL, its pages in logical order (at most `cap` written).  For tests and
 * tools.  Errors: EINVAL.
 */
int kvx_cache_agent(const kvx_cache *cache, int64_t agent, int32_t *cached_tokens, int32_t *page_ids,
                    int64_t cap);

/*
 * Host pages of `agent` in tokens (0 for an unknown agent) and, if `slots` is
 * non-NULL, their records in logical order (at most `cap` written).  For tests
 * and tools.  Errors: EINVAL.
 */
int kvx_cache_agent_host(const kvx_cache *cache, int64_t agent, int32_t *host_tokens, int32_t *slots,
                         int64_t cap);

/*
 * Make `agent` a member of `group` (any id), whose shared prefix is the first
 * `shared_tokens` tokens of every member's context, rounded down to whole pages.
 * The agent must be idle, hold no pages and belong to no group (a new agent);
 * every member of a group gives the same number of whole pages.
 * Errors: EINVAL (NULL cache, shared_tokens below one page, agent state,
 * a different span for an existing group).
 */
int kvx_cache_join(kvx_cache *cache, int64_t agent, int64_t group, int32_t shared_tokens);

/*
 * Shared pages of `group` in tokens (0 while its node is absent or the group is
 * unknown) and, if `page_ids` is non-NULL, the node's pages (at most `cap`).
 * For tests and tools.  Errors: EINVAL.
 */
int kvx_cache_group(const kvx_cache *cache, int64_t group, int32_t *shared_tokens, int32_t *page_ids,
                    int64_t cap);

/* Counters of the cache.  Errors: EINVAL. */
int kvx_cache_stats(const kvx_cache *cache, kvx_cache_counters *out);

#ifdef __cplusplus
}
#endif

#endif /* KVX_CACHE_H */
