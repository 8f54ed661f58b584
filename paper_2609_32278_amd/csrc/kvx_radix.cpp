// Token-content prefix cache over a kvx page pool: a radix tree of cached token
// sequences in whole pages, longest-prefix matching with shared inner nodes, and
// eviction of idle leaves by round-robin tail chunks (paper Section 3.2,
// Algorithm 1) or by least-recent whole leaves (Section 3.1).  The model and the
// C ABI are declared in include/kvx_radix.h.

#include <algorithm>
#include <limits>
#include <map>
#include <new>
#include <set>
#include <vector>

#include "kvx_cache.h"
#include "kvx_internal.h"
#include "kvx_radix.h"

using kvx::report;

namespace {

using PageKey = std::vector<int32_t>;  // the token ids of a node's first page

struct RNode {
  int64_t parent = -1;                  // -1: the root
  std::map<PageKey, int64_t> children;  // by first page
  std::vector<int32_t> tokens;          // the span, whole pages
  std::vector<int32_t> pages;           // one pool page per span page
  int64_t owner = -1;                   // agent whose request created the node
  int64_t stamp = 0;
  int32_t refs = 0;                     // running requests whose path holds the node
};

struct RAgent {
  bool active = false;
  std::vector<int64_t> path;   // pinned nodes of the running request, root side first
  std::vector<int32_t> temps;  // its pages the tree will not keep
};

// The outcome of walking the tree along a prompt.
struct Match {
  std::vector<int64_t> nodes;  // fully matched nodes, root side first
  int64_t partial = -1;        // a node matched over its first `partial_pages` pages only
  int64_t partial_pages = 0;
  int64_t pages = 0;           // matched pages in total
};

}  // namespace

struct kvx_radix {
  int64_t num_pages = 0;
  int32_t page_size = 0;
  int32_t chunk_pages = 0;
  int32_t policy = 0;
  std::set<int32_t> free_pages;               // handed out lowest id first
  std::map<int64_t, RNode> nodes;             // node id -> node; 0 is the root
  int64_t next_id = 1;
  std::map<int64_t, RAgent> agents;           // ordered by id: the round-robin order
  std::map<int64_t, std::set<int64_t>> owned; // agent -> the nodes it owns
  int64_t clock = 0;
  bool rr_started = false;
  int64_t rr_last = 0;                        // the agent that lost the last RR chunk
  int64_t evicted_pages = 0;
  int64_t evictions = 0;
};

namespace {

PageKey page_key(const int32_t* tokens, int ps) { return PageKey(tokens, tokens + ps); }

Match walk(const kvx_radix* t, const int32_t* tokens, int64_t whole) {
  const int ps = t->page_size;
  Match m;
  int64_t x = 0;
  while (m.pages < whole) {
    const RNode& nx = t->nodes.at(x);
    auto it = nx.children.find(page_key(tokens + m.pages * ps, ps));
    if (it == nx.children.end()) break;
    const RNode& c = t->nodes.at(it->second);
    const int64_t span = (int64_t)c.pages.size();
    int64_t k = 0;
    while (k < span && m.pages + k < whole &&
           std::equal(c.tokens.begin() + k * ps, c.tokens.begin() + (k + 1) * ps, tokens + (m.pages + k) * ps))
      k++;
    if (k == span) {
      m.nodes.push_back(it->second);
      m.pages += k;
      x = it->second;
      continue;
    }
    if (k > 0) {
      m.partial = it->second;
      m.partial_pages = k;
      m.pages += k;
    }
    break;
  }
  return m;
}

// Split node `id` after its first k pages: the node keeps them, a new child (same
// owner, stamp and pins) takes the rest and the old children.
int64_t split(kvx_radix* t, int64_t id, int64_t k) {
  const int ps = t->page_size;
  const int64_t tail_id = t->next_id++;
  RNode& n = t->nodes.at(id);
  RNode tail;
  tail.parent = id;
  tail.tokens.assign(n.tokens.begin() + k * ps, n.tokens.end());
  tail.pages.assign(n.pages.begin() + k, n.pages.end());
  tail.owner = n.owner;
  tail.stamp = n.stamp;
  tail.refs = n.refs;
  tail.children.swap(n.children);
  n.tokens.resize((size_t)(k * ps));
  n.pages.resize((size_t)k);
  n.children[page_key(tail.tokens.data(), ps)] = tail_id;
  for (auto& ch : tail.children) t->nodes.at(ch.second).parent = tail_id;
  t->owned[tail.owner].insert(tail_id);
  t->nodes.emplace(tail_id, std::move(tail));
  // running requests whose path crossed the whole node cross its tail too
  for (auto& a : t->agents) {
    std::vector<int64_t>& p = a.second.path;
    auto pos = std::find(p.begin(), p.end(), id);
    if (pos != p.end()) p.insert(pos + 1, tail_id);
  }
  return tail_id;
}

bool is_leaf(const kvx_radix* t, int64_t id) { return id != 0 && t->nodes.at(id).children.empty(); }

bool evictable(const kvx_radix* t, int64_t id) { return is_leaf(t, id) && t->nodes.at(id).refs == 0; }

// The agent's evictable leaf with the oldest stamp (ties: the older node), or -1.
int64_t oldest_leaf_of(const kvx_radix* t, int64_t agent) {
  auto it = t->owned.find(agent);
  if (it == t->owned.end()) return -1;
  int64_t best = -1;
  for (int64_t id : it->second) {
    if (!evictable(t, id)) continue;
    if (best < 0 || t->nodes.at(id).stamp < t->nodes.at(best).stamp) best = id;  // ids ascend
  }
  return best;
}

bool agent_active(const kvx_radix* t, int64_t agent) {
  auto it = t->agents.find(agent);
  return it != t->agents.end() && it->second.active;
}

// Drop the last k pages of leaf `id` (the whole leaf when k covers it).
void drop_tail(kvx_radix* t, int64_t id, int64_t k) {
  RNode& n = t->nodes.at(id);
  const int ps = t->page_size;
  const int64_t span = (int64_t)n.pages.size();
  for (int64_t i = span - k; i < span; i++) t->free_pages.insert(n.pages[(size_t)i]);
  if (k < span) {
    n.pages.resize((size_t)(span - k));
    n.tokens.resize((size_t)((span - k) * ps));
    return;
  }
  RNode& parent = t->nodes.at(n.parent);
  parent.children.erase(page_key(n.tokens.data(), ps));
  t->owned[n.owner].erase(id);
  if (t->owned[n.owner].empty()) t->owned.erase(n.owner);
  t->nodes.erase(id);
}

int64_t reclaim_rr(kvx_radix* t, int64_t M) {
  int64_t freed = 0;
  while (freed < M) {
    // Algorithm 1's queue: idle agents with an evictable suffix, in agent-id order
    // from the one after the agent that lost the last chunk
    std::vector<int64_t> ids;
    for (const auto& o : t->owned)
      if (!agent_active(t, o.first) && oldest_leaf_of(t, o.first) >= 0) ids.push_back(o.first);
    if (ids.empty()) break;
    size_t start = 0;
    if (t->rr_started) {
      start = (size_t)(std::upper_bound(ids.begin(), ids.end(), t->rr_last) - ids.begin());
      if (start == ids.size()) start = 0;
    }
    std::vector<int64_t> queue(ids.begin() + (ptrdiff_t)start, ids.end());
    queue.insert(queue.end(), ids.begin(), ids.begin() + (ptrdiff_t)start);
    size_t head = 0;
    while (freed < M && head < queue.size()) {
      const int64_t tau = queue[head++];
      const int64_t leaf = agent_active(t, tau) ? -1 : oldest_leaf_of(t, tau);  // eligibility, rechecked
      if (leaf < 0) continue;
      const int64_t k = std::min<int64_t>({(int64_t)t->chunk_pages, (int64_t)t->nodes.at(leaf).pages.size(),
                                           M - freed});
      drop_tail(t, leaf, k);
      freed += k;
      t->evicted_pages += k;
      t->evictions++;
      t->rr_started = true;
      t->rr_last = tau;
      if (oldest_leaf_of(t, tau) >= 0) queue.push_back(tau);
    }
  }
  return freed;
}

int64_t reclaim_lru(kvx_radix* t, int64_t M) {
  int64_t freed = 0;
  while (freed < M) {
    int64_t best = -1;
    for (const auto& n : t->nodes)
      if (evictable(t, n.first) && (best < 0 || n.second.stamp < t->nodes.at(best).stamp)) best = n.first;
    if (best < 0) break;
    const int64_t k = (int64_t)t->nodes.at(best).pages.size();
    drop_tail(t, best, k);
    freed += k;
    t->evicted_pages += k;
    t->evictions++;
  }
  return freed;
}

int check_tokens(const int32_t* tokens, int32_t n) {
  if (n < 1) return report(KVX_EINVAL, "n = %d must be >= 1", n);
  if (tokens == nullptr) return report(KVX_EINVAL, "tokens is NULL");
  return KVX_OK;
}

}  // namespace

extern "C" {

int kvx_radix_create(int64_t num_pages, int32_t page_size, int32_t chunk_tokens, int32_t policy,
                     kvx_radix** out) {
  if (out == nullptr) return report(KVX_EINVAL, "out is NULL");
  *out = nullptr;
  if (num_pages <= 0 || num_pages > (int64_t)std::numeric_limits<int32_t>::max())
    return report(KVX_EINVAL, "num_pages = %lld must be in [1, 2^31-1]", (long long)num_pages);
  if (page_size != kvx::kPageSize) return report(KVX_EUNSUPPORTED, "page_size %d (supported: 16)", page_size);
  if (chunk_tokens <= 0 || chunk_tokens % page_size != 0)
    return report(KVX_EINVAL, "chunk_tokens = %d must be a positive multiple of %d", chunk_tokens, page_size);
  if (policy != KVX_EVICT_LRU && policy != KVX_EVICT_RR) return report(KVX_EINVAL, "policy %d", policy);
  kvx_radix* t = new (std::nothrow) kvx_radix();
  if (t == nullptr) return report(KVX_ENOMEM, "tree allocation failed");
  try {
    for (int64_t i = 0; i < num_pages; i++) t->free_pages.insert(t->free_pages.end(), (int32_t)i);
    t->nodes.emplace(0, RNode());
  } catch (...) {
    delete t;
    return report(KVX_ENOMEM, "free list of %lld pages", (long long)num_pages);
  }
  t->num_pages = num_pages;
  t->page_size = page_size;
  t->chunk_pages = chunk_tokens / page_size;
  t->policy = policy;
  *out = t;
  return KVX_OK;
}

int kvx_radix_destroy(kvx_radix* tree) {
  delete tree;
  return KVX_OK;
}

int kvx_radix_begin(kvx_radix* t, int64_t agent, const int32_t* tokens, int32_t n, int32_t* prefix_len,
                    int32_t* page_ids, int64_t cap) {
  if (t == nullptr) return report(KVX_EINVAL, "tree is NULL");
  if (int rc = check_tokens(tokens, n)) return rc;
  if (prefix_len == nullptr || page_ids == nullptr) return report(KVX_EINVAL, "prefix_len and page_ids must be non-NULL");
  const int ps = t->page_size;
  const int64_t whole = n / ps, npages = ((int64_t)n + ps - 1) / ps;
  if (cap < npages) return report(KVX_EINVAL, "cap = %lld < %lld pages", (long long)cap, (long long)npages);
  if (agent_active(t, agent)) return report(KVX_EINVAL, "agent %lld already has a running request", (long long)agent);
  try {
    Match m = walk(t, tokens, whole);
    if (m.partial >= 0) {
      split(t, m.partial, m.partial_pages);
      m.nodes.push_back(m.partial);
    }
    const int64_t reuse = std::min<int64_t>(m.pages, ((int64_t)n - 1) / ps);
    RAgent& a = t->agents[agent];
    a.path = m.nodes;
    a.temps.clear();
    a.active = true;
    const int64_t now = ++t->clock;
    for (int64_t id : a.path) {
      RNode& x = t->nodes.at(id);
      x.refs++;
      x.stamp = now;
    }
    const int64_t need = npages - reuse;
    if ((int64_t)t->free_pages.size() < need) {
      const int64_t M = need - (int64_t)t->free_pages.size();
      if (t->policy == KVX_EVICT_RR) reclaim_rr(t, M);
      else reclaim_lru(t, M);
    }
    if ((int64_t)t->free_pages.size() < need) {
      for (int64_t id : a.path) t->nodes.at(id).refs--;
      a.path.clear();
      a.active = false;
      return report(KVX_ENOMEM, "request of %d tokens needs %lld pages; %lld free after reclaiming every idle page", n,
                    (long long)need, (long long)t->free_pages.size());
    }
    std::vector<int32_t> fresh((size_t)need);
    for (int64_t i = 0; i < need; i++) {
      fresh[(size_t)i] = *t->free_pages.begin();
      t->free_pages.erase(t->free_pages.begin());
    }
    // page table: the reused tree pages, then the fresh ones
    int64_t j = 0;
    for (int64_t id : m.nodes)
      for (int32_t pg : t->nodes.at(id).pages)
        if (j < reuse) page_ids[j++] = pg;
    for (int64_t i = 0; i < need; i++) page_ids[reuse + i] = fresh[(size_t)i];
    // the prompt's whole pages past the match become the agent's new leaf
    if (whole > m.pages) {
      const int64_t parent = m.nodes.empty() ? 0 : m.nodes.back();
      const int64_t id = t->next_id++;
      RNode leaf;
      leaf.parent = parent;
      leaf.tokens.assign(tokens + m.pages * ps, tokens + whole * ps);
      leaf.pages.assign(fresh.begin() + (m.pages - reuse), fresh.begin() + (whole - reuse));
      leaf.owner = agent;
      leaf.stamp = now;
      leaf.refs = 1;
      t->nodes.at(parent).children[page_key(leaf.tokens.data(), ps)] = id;
      t->nodes.emplace(id, std::move(leaf));
      t->owned[agent].insert(id);
      a.path.push_back(id);
    }
    // recomputed pages the tree already holds, and a partial last page
    for (int64_t lp = reuse; lp < std::min(m.pages, npages); lp++) a.temps.push_back(fresh[(size_t)(lp - reuse)]);
    if (npages > whole && npages > m.pages) a.temps.push_back(fresh.back());
    *prefix_len = (int32_t)(reuse * ps);
  } catch (const std::bad_alloc&) {
    return report(KVX_ENOMEM, "host allocation failed");
  }
  return KVX_OK;
}

int kvx_radix_end(kvx_radix* t, int64_t agent) {
  if (t == nullptr) return report(KVX_EINVAL, "tree is NULL");
  auto it = t->agents.find(agent);
  if (it == t->agents.end() || !it->second.active)
    return report(KVX_EINVAL, "agent %lld has no running request", (long long)agent);
  RAgent& a = it->second;
  const int64_t now = ++t->clock;
  for (int64_t id : a.path) {
    RNode& x = t->nodes.at(id);
    x.refs--;
    x.stamp = now;
  }
  for (int32_t pg : a.temps) t->free_pages.insert(pg);
  a.path.clear();
  a.temps.clear();
  a.active = false;
  return KVX_OK;
}

int kvx_radix_complete(kvx_radix* t, int64_t agent) {
  if (t == nullptr) return report(KVX_EINVAL, "tree is NULL");
  if (agent_active(t, agent)) return report(KVX_EINVAL, "agent %lld has a running request", (long long)agent);
  for (;;) {
    auto it = t->owned.find(agent);
    if (it == t->owned.end()) break;
    int64_t leaf = -1;
    for (int64_t id : it->second)
      if (evictable(t, id)) {
        leaf = id;
        break;
      }
    if (leaf < 0) break;
    drop_tail(t, leaf, (int64_t)t->nodes.at(leaf).pages.size());
  }
  return KVX_OK;
}

int kvx_radix_match(const kvx_radix* t, const int32_t* tokens, int32_t n, int32_t* matched_tokens,
                    int32_t* page_ids, int64_t cap) {
  if (t == nullptr) return report(KVX_EINVAL, "tree is NULL");
  if (int rc = check_tokens(tokens, n)) return rc;
  if (matched_tokens == nullptr) return report(KVX_EINVAL, "matched_tokens is NULL");
  const Match m = walk(t, tokens, n / t->page_size);
  *matched_tokens = (int32_t)(m.pages * t->page_size);
  if (page_ids != nullptr) {
    int64_t j = 0;
    std::vector<int64_t> ids = m.nodes;
    if (m.partial >= 0) ids.push_back(m.partial);
    for (int64_t id : ids) {
      const RNode& x = t->nodes.at(id);
      const int64_t take = id == m.partial ? m.partial_pages : (int64_t)x.pages.size();
      for (int64_t i = 0; i < take && j < cap; i++) page_ids[j++] = x.pages[(size_t)i];
    }
  }
  return KVX_OK;
}

int kvx_radix_stats(const kvx_radix* t, kvx_radix_counters* out) {
  if (t == nullptr || out == nullptr) return report(KVX_EINVAL, "tree and out must be non-NULL");
  kvx_radix_counters c{};
  c.num_pages = t->num_pages;
  c.free_pages = (int64_t)t->free_pages.size();
  for (const auto& n : t->nodes) {
    if (n.first == 0) continue;
    c.nodes++;
    c.cached_pages += (int64_t)n.second.pages.size();
    if (n.second.children.empty()) c.leaves++;
  }
  for (const auto& a : t->agents) {
    c.temp_pages += (int64_t)a.second.temps.size();
    if (a.second.active) c.active++;
  }
  c.evicted_pages = t->evicted_pages;
  c.evictions = t->evictions;
  *out = c;
  return KVX_OK;
}

}  // extern "C"
