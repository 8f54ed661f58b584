/*
 * kvx_radix.h -- a token-content prefix cache over the kvx page pool: a radix
 * tree of cached token sequences with longest-prefix matching, shared inner
 * nodes, and eviction of idle leaves by round-robin tail chunks (paper Section
 * 3.2, Algorithm 1) or by least-recent whole leaves (the LRU baseline of
 * Sections 3.1 and 4).
 *
 * The model (Section 2, "Prefix caching for multi-turn agents": requests reuse
 * the KV of their longest matching prefix in a radix tree whose nodes hold
 * variable-length spans; Section 3.1: active nodes cannot be reclaimed, and
 * eviction starts at idle leaves and exposes their parents).
 *   - The tree indexes whole pages: a node holds a span of page_size-token pages
 *     of token ids and one pool page per span page.  Siblings differ in their
 *     first page; a match compares whole pages and stops at the first page that
 *     differs (or at the prompt's last whole page).
 *   - A request (one agent's turn) of n tokens reuses the matched pages up to the
 *     last whole page before its final token (at least one token is computed):
 *       prefix_len = page_size * min(matched pages, floor((n - 1) / page_size)).
 *     Its page table: reused tree pages, then fresh pages for the rest.  The
 *     prompt's whole pages past the match become a new leaf (owned by the
 *     agent) under the match point, splitting a node whose span the match ends
 *     inside; fresh pages of already cached whole pages (past the reuse limit)
 *     and of a partial last page are temporary and freed at the request's end.
 *   - Every node on a running request's path is pinned.  A request start and end
 *     stamp every node of its path with the logical clock (one tick per start
 *     and per end): nodes touched together share a stamp (the recency
 *     synchronization of Section 3.1).
 *   - A node belongs to the trajectory (agent) whose request created it; a split
 *     keeps the owner.  An agent's evictable suffix is its leaves that no running
 *     request pins.
 * Reclamation of M pages when a request start finds too few free:
 *   KVX_EVICT_RR   Algorithm 1: idle agents with an evictable suffix form a queue
 *                  in agent-id order, starting after the agent that lost the last
 *                  chunk of any earlier reclamation.  The front agent loses one
 *                  tail chunk -- the last min(chunk, leaf pages, M - freed) pages
 *                  of its evictable leaf with the oldest stamp (ties: the older
 *                  node) -- and goes to the back while it still has an evictable
 *                  suffix; eligibility is rechecked at every pop.  A leaf emptied
 *                  by a chunk is removed, which may expose its parent as a leaf
 *                  of the parent's owner.  If the queue runs empty before M pages
 *                  are freed, a new queue is formed (exposed parents of agents
 *                  that were not queued become candidates).
 *   KVX_EVICT_LRU  repeatedly removes the whole unpinned leaf with the oldest
 *                  stamp (ties: the older node), exposing its parent.
 * Completion signal (Section 3.2): kvx_radix_complete frees an idle agent's
 * unshared cache at once -- its unpinned leaves, repeatedly, as far as they are
 * its own.
 *
 * Conventions as in kvx_cache.h: synchronous host code, KVX_OK or a kvx_status
 * code (kvx_last_error() describes the failure), not thread-safe for one tree,
 * page ids index a kvx pool of the same num_pages, and the tree never touches the
 * pool's memory.  Free pages are handed out lowest id first.
 */
#ifndef KVX_RADIX_H
#define KVX_RADIX_H

#include <stdint.h>

#include "kvx.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kvx_radix kvx_radix; /* opaque; owned by the library */

typedef struct {
    int64_t num_pages;     /* pool pages managed */
    int64_t free_pages;    /* pages owned by nobody */
    int64_t cached_pages;  /* pages held by tree nodes */
    int64_t temp_pages;    /* running requests' pages that the tree will not keep */
    int64_t nodes;         /* tree nodes, the root excluded */
    int64_t leaves;        /* nodes without children */
    int64_t evicted_pages; /* pages reclaimed by eviction since creation */
    int64_t evictions;     /* eviction steps (RR chunks or LRU leaves) since creation */
    int32_t active;        /* running requests */
    int32_t reserved;
} kvx_radix_counters;

/*
 * Create a tree over `num_pages` pages of `page_size` tokens.
 *   page_size     16 (the pool's page size).
 *   chunk_tokens  RR tail-chunk size in tokens, a positive multiple of page_size
 *                 (the paper evaluates 1024); checked but unused by LRU.
 *   policy        KVX_EVICT_LRU or KVX_EVICT_RR (kvx_cache.h).
 * Errors: EINVAL (sizes, policy, out NULL), EUNSUPPORTED (page_size), ENOMEM.
 */
int kvx_radix_create(int64_t num_pages, int32_t page_size, int32_t chunk_tokens, int32_t policy,
                     kvx_radix **out);

/* Free a tree.  NULL is a no-op. */
int kvx_radix_destroy(kvx_radix *tree);

/*
 * Start a request of `agent` over tokens[0 .. n), n >= 1 (host token ids): match,
 * pin, reclaim if needed, allocate, insert (see the model above).  On success
 * *prefix_len holds the reused tokens and page_ids[0 .. ceil(n / page_size)) the
 * request's page table, ready for store_kv / extend_attention with
 * P = *prefix_len and E = n - *prefix_len; the agent is running.
 *   page_ids, cap  host buffer of cap >= ceil(n / page_size) entries.
 * Errors: EINVAL (agent already running, n < 1, cap, NULL pointers), ENOMEM (too
 * few pages even after reclaiming everything evictable: pages evicted so far stay
 * evicted, nothing is inserted and the agent stays idle).
 */
int kvx_radix_begin(kvx_radix *tree, int64_t agent, const int32_t *tokens, int32_t n, int32_t *prefix_len,
                    int32_t *page_ids, int64_t cap);

/* End `agent`'s running request: unpin and stamp its path, free its temporary
 * pages.  Errors: EINVAL (not running). */
int kvx_radix_end(kvx_radix *tree, int64_t agent);

/* Completion signal for an idle `agent` (see above).  Errors: EINVAL (running). */
int kvx_radix_complete(kvx_radix *tree, int64_t agent);

/*
 * Longest cached prefix of tokens[0 .. n) in whole pages, in tokens (no reuse
 * limit, no stamps, no pins): a read-only probe for tests and tools.  If
 * page_ids is non-NULL, the matched pages go there (at most cap).  Errors: EINVAL.
 */
int kvx_radix_match(const kvx_radix *tree, const int32_t *tokens, int32_t n, int32_t *matched_tokens,
                    int32_t *page_ids, int64_t cap);

/* Counters.  Errors: EINVAL. */
int kvx_radix_stats(const kvx_radix *tree, kvx_radix_counters *out);

#ifdef __cplusplus
}
#endif

#endif /* KVX_RADIX_H */
