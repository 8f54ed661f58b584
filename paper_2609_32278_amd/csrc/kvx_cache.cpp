// Host-side prefix cache for multi-turn agents: page allocation over a kvx pool
// and eviction of idle agents' histories, either by round-robin tail chunks
// (paper Section 3.2, Algorithm 1) or by least-recent whole leaf nodes (the LRU
// baseline, Section 3.1), optionally into a host tier of spilled pages that a
// returning agent reloads (the paper's future work, Section 6).  The C ABI and
// the model are declared in include/kvx_cache.h.

#include <algorithm>
#include <deque>
#include <limits>
#include <map>
#include <new>
#include <vector>

#include "kvx_cache.h"
#include "kvx_internal.h"

namespace {

struct CacheNode {
  std::vector<int32_t> pages;  // logical order
};

struct CacheAgent {
  std::vector<CacheNode> nodes;  // root .. leaf; never empty nodes
  int64_t pages = 0;             // cached pages (sum over nodes)
  int64_t stamp = 0;             // time stamp shared by every node of the path
  bool active = false;
  int32_t prompt_len = 0;        // running turn
  std::vector<int32_t> turn;     // pages allocated to the running turn
  std::deque<int32_t> host;      // host records continuing the device pages, nearest first
  bool in_group = false;
  int64_t group = 0;
  int64_t turn_start = 0;        // logical page of the running turn's first page
};

// A shared prefix (system prompt) of a group of agents: one node of S whole
// pages, present or absent as a whole, read by every member's page table.
struct CacheGroup {
  int64_t S = 0;
  bool present = false;
  std::vector<int32_t> pages;
  int64_t stamp = 0;
  std::vector<int64_t> members;
};

struct FifoEntry {
  int32_t rec;
  uint32_t gen;  // generation of the record when it was spilled into
};

}  // namespace

struct kvx_cache {
  int64_t num_pages = 0;
  int32_t page_size = 0;
  int32_t chunk_pages = 0;
  int32_t policy = 0;
  std::vector<int32_t> free_pages;       // stack; the next page handed out is at the back
  std::map<int64_t, CacheAgent> agents;  // ordered by id: the round-robin order
  std::map<int64_t, CacheGroup> groups;
  int64_t group_pages = 0;               // pages of present group nodes
  int64_t clock = 0;
  bool rr_has_last = false;
  int64_t rr_last = 0;  // agent that lost the last RR chunk
  int64_t evicted_pages = 0;
  int64_t evictions = 0;
  int64_t tier_width = 0;  // recency tiers of the round robin (0: off)
  // host tier
  int64_t host_pages = 0;
  std::vector<int32_t> host_free;     // stack of free records
  std::deque<FifoEntry> host_fifo;    // spills, oldest first (entries of freed records are stale)
  std::vector<int64_t> rec_owner;     // agent of each live record
  std::vector<uint32_t> rec_gen;      // bumped at every allocation of the record
  std::vector<uint8_t> rec_live;
  int64_t host_used = 0, spilled = 0, reloaded = 0, host_dropped = 0;
  std::vector<int32_t> mv_spill_pages, mv_spill_slots, mv_reload_pages, mv_reload_slots;
  // per turn start: FIFO entries before fifo_scan belong to the agent inside the
  // turn (pinned for the whole call); rec_call / rec_move locate a record's spill
  // in this call's move list
  size_t fifo_scan = 0;
  uint64_t call = 0;
  std::vector<uint64_t> rec_call;
  std::vector<int32_t> rec_move;
};

namespace {

using kvx::report;

void release_pages(kvx_cache* c, const int32_t* p, size_t n) {
  for (size_t i = n; i-- > 0;) c->free_pages.push_back(p[i]);
}

// Drop the last `n` cached pages of an agent (n <= agent pages), leaf first.
void drop_tail(kvx_cache* c, CacheAgent& a, int64_t n) {
  while (n > 0) {
    CacheNode& leaf = a.nodes.back();
    const int64_t k = std::min<int64_t>(n, (int64_t)leaf.pages.size());
    const size_t keep = leaf.pages.size() - (size_t)k;
    release_pages(c, leaf.pages.data() + keep, (size_t)k);
    leaf.pages.resize(keep);
    if (leaf.pages.empty()) a.nodes.pop_back();
    a.pages -= k;
    n -= k;
  }
}

void free_record(kvx_cache* c, int32_t rec) {
  c->rec_live[(size_t)rec] = 0;
  c->host_free.push_back(rec);
  c->host_used--;
}

void drop_host(kvx_cache* c, CacheAgent& a, size_t keep) {
  while (a.host.size() > keep) {
    free_record(c, a.host.back());
    a.host.pop_back();
  }
}

// A group node is a leaf while no member is inside a turn and no member holds
// private or host pages.
bool group_leaf(const kvx_cache* c, const CacheGroup& g) {
  if (!g.present) return false;
  for (int64_t m : g.members) {
    const CacheAgent& a = c->agents.find(m)->second;
    if (a.active || a.pages > 0 || !a.host.empty()) return false;
  }
  return true;
}

// Evict a group node whole (never spilled).
int64_t evict_group(kvx_cache* c, CacheGroup& g) {
  const int64_t n = (int64_t)g.pages.size();
  release_pages(c, g.pages.data(), g.pages.size());
  g.pages.clear();
  g.present = false;
  c->group_pages -= n;
  c->evicted_pages += n;
  c->evictions++;
  return n;
}

// A record for a spill of `owner`'s page: a free one, else the oldest live record
// whose owner is idle is dropped (it is always that owner's farthest host page);
// -1 if every record belongs to an agent inside a turn.
int32_t take_record(kvx_cache* c, int64_t owner) {
  int32_t rec = -1;
  if (!c->host_free.empty()) {
    rec = c->host_free.back();
    c->host_free.pop_back();
  } else {
    for (auto it = c->host_fifo.begin() + (std::ptrdiff_t)c->fifo_scan; it != c->host_fifo.end();) {
      const int32_t r = it->rec;
      if (!c->rec_live[(size_t)r] || c->rec_gen[(size_t)r] != it->gen) {
        it = c->host_fifo.erase(it);  // freed since
        continue;
      }
      CacheAgent& o = c->agents.find(c->rec_owner[(size_t)r])->second;
      if (o.active) {  // the agent inside the turn: stays active for the rest of the call
        ++it;
        c->fifo_scan++;
        continue;
      }
      // r is o's farthest host page (one agent's spills enter the FIFO farthest
      // page first); were it not, the pages past it would go too, keeping o's
      // history free of gaps
      c->host_fifo.erase(it);
      while (!o.host.empty() && o.host.back() != r) {
        free_record(c, o.host.back());
        o.host.pop_back();
        c->host_dropped++;
      }
      o.host.pop_back();
      c->host_used--;
      rec = r;
      // a record spilled into earlier in this same call: that spill is void (its
      // page is simply dropped); its move is struck out and removed at the end
      if (c->rec_call[(size_t)r] == c->call) {
        c->mv_spill_pages[(size_t)c->rec_move[(size_t)r]] = -1;
        c->spilled--;
      } else {
        c->host_dropped++;
      }
      break;
    }
    if (rec < 0) return -1;
  }
  c->rec_live[(size_t)rec] = 1;
  c->rec_gen[(size_t)rec]++;
  c->rec_owner[(size_t)rec] = owner;
  c->host_used++;
  c->host_fifo.push_back(FifoEntry{rec, c->rec_gen[(size_t)rec]});
  if ((int64_t)c->host_fifo.size() > 2 * c->host_pages + 64) {  // drop the entries of freed records
    std::deque<FifoEntry> live;
    for (const FifoEntry& e : c->host_fifo)
      if (c->rec_live[(size_t)e.rec] && c->rec_gen[(size_t)e.rec] == e.gen) live.push_back(e);
    c->host_fifo.swap(live);
    c->fifo_scan = 0;  // recounted by the next walk
  }
  return rec;
}

// Evict the last n device pages of agent `id`: freed, and spilled to the host
// tier (farthest page first) when there is one.
void evict_tail(kvx_cache* c, int64_t id, CacheAgent& a, int64_t n) {
  std::vector<int32_t> pages;
  if (c->host_pages > 0) {
    for (auto nd = a.nodes.rbegin(); nd != a.nodes.rend() && (int64_t)pages.size() < n; ++nd)
      for (auto pg = nd->pages.rbegin(); pg != nd->pages.rend() && (int64_t)pages.size() < n; ++pg)
        pages.push_back(*pg);  // farthest first
  }
  drop_tail(c, a, n);
  for (int32_t pg : pages) {
    const int32_t rec = take_record(c, id);
    if (rec < 0) continue;  // dropped: the agent holds no host pages past it
    a.host.push_front(rec);
    c->rec_call[(size_t)rec] = c->call;
    c->rec_move[(size_t)rec] = (int32_t)c->mv_spill_pages.size();
    c->mv_spill_pages.push_back(pg);
    c->mv_spill_slots.push_back(rec);
    c->spilled++;
  }
}

// LRU: whole leaf nodes, oldest time stamp first (ties: smaller id), idle agents only.
int64_t evict_lru(kvx_cache* c, int64_t need) {
  int64_t freed = 0;
  while (freed < need) {
    CacheAgent* best = nullptr;
    int64_t best_id = 0;
    for (auto& kv : c->agents) {
      CacheAgent& a = kv.second;
      if (a.active || a.nodes.empty()) continue;
      if (best == nullptr || a.stamp < best->stamp) {  // map order breaks ties by id
        best = &a;
        best_id = kv.first;
      }
    }
    CacheGroup* leaf = nullptr;  // a group node older than every agent leaf goes first
    for (auto& kv : c->groups)
      if (group_leaf(c, kv.second) && (leaf == nullptr || kv.second.stamp < leaf->stamp) &&
          (best == nullptr || kv.second.stamp < best->stamp))
        leaf = &kv.second;
    if (leaf != nullptr) {
      freed += evict_group(c, *leaf);
      continue;
    }
    if (best == nullptr) break;
    const int64_t n = (int64_t)best->nodes.back().pages.size();
    evict_tail(c, best_id, *best, n);
    freed += n;
    c->evicted_pages += n;
    c->evictions++;
  }
  return freed;
}

// Algorithm 1: one queue of idle agents with evictable pages, in id order starting
// after the agent that lost the previous chunk; one tail chunk per visit.
// Algorithm 1 over the idle agents `ids` (ascending id order): one queue starting
// after the agent that lost the previous chunk, one tail chunk per visit, until
// `need` pages are freed in total or the queue is empty.
int64_t round_robin(kvx_cache* c, const std::vector<int64_t>& ids, int64_t need, int64_t freed) {
  std::deque<int64_t> q;
  const size_t start = c->rr_has_last
                           ? (size_t)(std::upper_bound(ids.begin(), ids.end(), c->rr_last) - ids.begin())
                           : 0;
  for (size_t i = start; i < ids.size(); i++) q.push_back(ids[i]);
  for (size_t i = 0; i < start; i++) q.push_back(ids[i]);
  while (freed < need && !q.empty()) {
    const int64_t id = q.front();
    q.pop_front();
    auto it = c->agents.find(id);
    if (it == c->agents.end()) continue;
    CacheAgent& a = it->second;
    if (a.active || a.pages == 0) continue;  // eligibility rechecked at every pop
    // SelectTailChunk: a suffix of the leaf node, at most one chunk and at most
    // what is still to be reclaimed
    const int64_t n = std::min<int64_t>({(int64_t)c->chunk_pages, (int64_t)a.nodes.back().pages.size(),
                                         need - freed});
    evict_tail(c, id, a, n);
    freed += n;
    c->evicted_pages += n;
    c->evictions++;
    c->rr_has_last = true;
    c->rr_last = id;
    if (a.pages > 0) q.push_back(id);
  }
  return freed;
}

// Round-robin reclamation; with recency tiers, tier by tier from the oldest
// (age = clock - stamp, tier = age / tier_width), round robin within each.
int64_t evict_rr(kvx_cache* c, int64_t need) {
  std::map<int64_t, std::vector<int64_t>> tiers;  // tier -> idle agents holding pages, id order
  for (const auto& kv : c->agents) {
    const CacheAgent& a = kv.second;
    if (a.active || a.pages == 0) continue;
    const int64_t tier = c->tier_width > 0 ? (c->clock - a.stamp) / c->tier_width : 0;
    tiers[tier].push_back(kv.first);
  }
  int64_t freed = 0;
  for (auto t = tiers.rbegin(); t != tiers.rend() && freed < need; ++t) freed = round_robin(c, t->second, need, freed);
  if (freed < need) {  // group nodes, parents of every member's path, oldest first
    std::vector<std::pair<int64_t, int64_t>> leaves;  // (stamp, group)
    for (auto& kv : c->groups)
      if (group_leaf(c, kv.second)) leaves.emplace_back(kv.second.stamp, kv.first);
    std::sort(leaves.begin(), leaves.end());
    for (const auto& l : leaves) {
      if (freed >= need) break;
      freed += evict_group(c, c->groups[l.second]);
    }
  }
  return freed;
}

int64_t div_up(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

extern "C" {

int kvx_cache_create(int64_t num_pages, int32_t page_size, int32_t chunk_tokens, int32_t policy,
                     kvx_cache** out) {
  return kvx_cache_create_tiered(num_pages, 0, page_size, chunk_tokens, policy, out);
}

int kvx_cache_create_tiered(int64_t num_pages, int64_t host_pages, int32_t page_size, int32_t chunk_tokens,
                            int32_t policy, kvx_cache** out) {
  if (out == nullptr) return report(KVX_EINVAL, "out is NULL");
  *out = nullptr;
  if (num_pages <= 0 || num_pages > (int64_t)std::numeric_limits<int32_t>::max())
    return report(KVX_EINVAL, "num_pages = %lld must be in [1, 2^31-1]", (long long)num_pages);
  if (page_size != kvx::kPageSize) return report(KVX_EUNSUPPORTED, "page_size %d (supported: 16)", page_size);
  if (chunk_tokens <= 0 || chunk_tokens % page_size != 0)
    return report(KVX_EINVAL, "chunk_tokens = %d must be a positive multiple of %d", chunk_tokens, page_size);
  if (policy != KVX_EVICT_LRU && policy != KVX_EVICT_RR) return report(KVX_EINVAL, "policy %d", policy);
  if (host_pages < 0 || host_pages > (int64_t)std::numeric_limits<int32_t>::max())
    return report(KVX_EINVAL, "host_pages = %lld must be in [0, 2^31-1]", (long long)host_pages);
  kvx_cache* c = new (std::nothrow) kvx_cache();
  if (c == nullptr) return report(KVX_ENOMEM, "cache allocation failed");
  try {
    c->free_pages.resize((size_t)num_pages);
    c->host_free.resize((size_t)host_pages);
    c->rec_owner.assign((size_t)host_pages, 0);
    c->rec_gen.assign((size_t)host_pages, 0);
    c->rec_live.assign((size_t)host_pages, 0);
    c->rec_call.assign((size_t)host_pages, 0);
    c->rec_move.assign((size_t)host_pages, 0);
  } catch (...) {
    delete c;
    return report(KVX_ENOMEM, "free lists of %lld pages and %lld records", (long long)num_pages,
                  (long long)host_pages);
  }
  for (int64_t i = 0; i < num_pages; i++) c->free_pages[(size_t)i] = (int32_t)(num_pages - 1 - i);  // page 0 first
  for (int64_t i = 0; i < host_pages; i++) c->host_free[(size_t)i] = (int32_t)(host_pages - 1 - i);
  c->host_pages = host_pages;
  c->num_pages = num_pages;
  c->page_size = page_size;
  c->chunk_pages = chunk_tokens / page_size;
  c->policy = policy;
  *out = c;
  return KVX_OK;
}

int kvx_cache_set_recency_tiers(kvx_cache* c, int64_t tier_width) {
  if (c == nullptr) return report(KVX_EINVAL, "cache is NULL");
  if (tier_width < 0) return report(KVX_EINVAL, "tier_width = %lld must be >= 0", (long long)tier_width);
  if (c->policy != KVX_EVICT_RR) return report(KVX_EINVAL, "recency tiers apply to KVX_EVICT_RR only");
  c->tier_width = tier_width;
  return KVX_OK;
}

int kvx_cache_destroy(kvx_cache* c) {
  delete c;
  return KVX_OK;
}

static int begin_turn(kvx_cache* c, int64_t agent, int32_t prompt_len, int32_t* prefix_len, int32_t* page_ids,
                      int64_t cap, kvx_cache_moves* moves) {
  if (c == nullptr || prefix_len == nullptr || page_ids == nullptr)
    return report(KVX_EINVAL, "cache, prefix_len and page_ids must be non-NULL");
  if (moves == nullptr && c->host_pages > 0)
    return report(KVX_EINVAL, "a cache with a host tier starts turns with kvx_cache_begin_turn_tiered");
  if (prompt_len < 1) return report(KVX_EINVAL, "prompt_len = %d must be >= 1", prompt_len);
  const int64_t S = c->page_size;
  const int64_t n_total = div_up(prompt_len, S);
  if (cap < n_total) return report(KVX_EINVAL, "page_ids holds %lld entries, the prompt needs %lld", (long long)cap,
                                   (long long)n_total);
  auto found = c->agents.find(agent);
  if (found != c->agents.end() && found->second.active)
    return report(KVX_EINVAL, "agent %lld is already inside a turn", (long long)agent);
  c->mv_spill_pages.clear();
  c->mv_spill_slots.clear();
  c->mv_reload_pages.clear();
  c->mv_reload_slots.clear();
  c->fifo_scan = 0;
  c->call++;
  CacheAgent& a = c->agents[agent];
  a.stamp = ++c->clock;  // matching the prefix touches every node of the path
  CacheGroup* g = a.in_group ? &c->groups[a.group] : nullptr;
  if (g != nullptr) g->stamp = a.stamp;
  // reuse the group's shared pages, then device pages, then host pages, up to the
  // last whole page before the final token
  const int64_t limit = (prompt_len - 1) / S;
  const int64_t gp = (g != nullptr && g->present) ? g->S : 0;
  const int64_t reuse_pages = std::min<int64_t>(gp + a.pages + (int64_t)a.host.size(), limit);
  int64_t used_group = gp;
  if (reuse_pages < gp) {  // the prompt ends inside the shared span
    used_group = reuse_pages;
    drop_host(c, a, 0);
    drop_tail(c, a, a.pages);
  } else if (reuse_pages - gp < a.pages) {
    drop_host(c, a, 0);
    drop_tail(c, a, a.pages - (reuse_pages - gp));
  } else {
    drop_host(c, a, (size_t)(reuse_pages - gp - a.pages));
  }
  const int64_t reload = (int64_t)a.host.size();
  a.turn_start = used_group + a.pages;
  const int64_t need = n_total - a.turn_start;  // reloaded pages + the suffix's pages
  a.active = true;  // pinned (with its host records) while this turn allocates
  if ((int64_t)c->free_pages.size() < need) {
    const int64_t want = need - (int64_t)c->free_pages.size();
    if (c->policy == KVX_EVICT_RR) evict_rr(c, want);
    else evict_lru(c, want);
  }
  auto fill_moves = [&]() {
    if (moves == nullptr) return;
    size_t w = 0;  // drop the struck-out (void) spills
    for (size_t i = 0; i < c->mv_spill_pages.size(); i++)
      if (c->mv_spill_pages[i] >= 0) {
        c->mv_spill_pages[w] = c->mv_spill_pages[i];
        c->mv_spill_slots[w] = c->mv_spill_slots[i];
        w++;
      }
    c->mv_spill_pages.resize(w);
    c->mv_spill_slots.resize(w);
    moves->spill_pages = c->mv_spill_pages.data();
    moves->spill_slots = c->mv_spill_slots.data();
    moves->reload_pages = c->mv_reload_pages.data();
    moves->reload_slots = c->mv_reload_slots.data();
    moves->n_spill = (int64_t)c->mv_spill_pages.size();
    moves->n_reload = (int64_t)c->mv_reload_pages.size();
  };
  if ((int64_t)c->free_pages.size() < need) {
    a.active = false;
    fill_moves();
    return report(KVX_ENOMEM, "agent %lld: %lld pages needed, %lld free after evicting every idle page",
                  (long long)agent, (long long)need, (long long)c->free_pages.size());
  }
  a.turn.clear();
  a.turn.reserve((size_t)need);
  for (int64_t i = 0; i < need; i++) {
    a.turn.push_back(c->free_pages.back());
    c->free_pages.pop_back();
  }
  for (int64_t j = 0; j < reload; j++) {
    c->mv_reload_pages.push_back(a.turn[(size_t)j]);
    c->mv_reload_slots.push_back(a.host[(size_t)j]);
  }
  drop_host(c, a, 0);
  c->reloaded += reload;
  a.prompt_len = prompt_len;
  int64_t j = 0;
  for (int64_t i = 0; i < used_group; i++) page_ids[j++] = g->pages[(size_t)i];
  for (const CacheNode& nd : a.nodes)
    for (int32_t pg : nd.pages) page_ids[j++] = pg;
  for (int32_t pg : a.turn) page_ids[j++] = pg;
  *prefix_len = (int32_t)(reuse_pages * S);
  fill_moves();
  return KVX_OK;
}

int kvx_cache_begin_turn(kvx_cache* c, int64_t agent, int32_t prompt_len, int32_t* prefix_len, int32_t* page_ids,
                         int64_t cap) {
  return begin_turn(c, agent, prompt_len, prefix_len, page_ids, cap, nullptr);
}

int kvx_cache_begin_turn_tiered(kvx_cache* c, int64_t agent, int32_t prompt_len, int32_t* prefix_len,
                                int32_t* page_ids, int64_t cap, kvx_cache_moves* moves) {
  if (moves == nullptr) return report(KVX_EINVAL, "moves is NULL");
  *moves = kvx_cache_moves{};
  return begin_turn(c, agent, prompt_len, prefix_len, page_ids, cap, moves);
}

int kvx_cache_end_turn(kvx_cache* c, int64_t agent) {
  if (c == nullptr) return report(KVX_EINVAL, "cache is NULL");
  auto it = c->agents.find(agent);
  if (it == c->agents.end() || !it->second.active)
    return report(KVX_EINVAL, "agent %lld is not inside a turn", (long long)agent);
  CacheAgent& a = it->second;
  // whole pages of the prompt stay cached; a partial last page is freed.  The turn
  // holds logical pages [turn_start, turn_start + turn.size()).
  const int64_t whole = a.prompt_len / c->page_size;
  int64_t keep_from = 0, keep_to = std::max<int64_t>(0, whole - a.turn_start);  // turn indices of the new node
  if (a.in_group) {
    CacheGroup& g = c->groups[a.group];
    int64_t donated = 0;
    if (!g.present && whole >= g.S) {  // the turn computed the shared span: it becomes the group node
      g.pages.assign(a.turn.begin(), a.turn.begin() + g.S);
      g.present = true;
      c->group_pages += g.S;
      donated = g.S;
    }
    if (g.present) {
      keep_from = std::max<int64_t>(g.S, a.turn_start) - a.turn_start;  // copies of the span are freed
      if (keep_from > keep_to) keep_from = keep_to;
    } else {
      keep_from = keep_to = 0;  // no private pages without the group node
    }
    if (keep_from > donated) release_pages(c, a.turn.data() + donated, (size_t)(keep_from - donated));
  }
  CacheNode nd;
  nd.pages.assign(a.turn.begin() + keep_from, a.turn.begin() + keep_to);
  if ((size_t)keep_to < a.turn.size()) release_pages(c, a.turn.data() + keep_to, a.turn.size() - (size_t)keep_to);
  if (!nd.pages.empty()) {
    a.pages += (int64_t)nd.pages.size();
    a.nodes.push_back(std::move(nd));
  }
  a.turn.clear();
  a.active = false;
  a.stamp = ++c->clock;  // inserting the turn's pages touches the whole path
  if (a.in_group) c->groups[a.group].stamp = a.stamp;
  return KVX_OK;
}

int kvx_cache_complete(kvx_cache* c, int64_t agent) {
  if (c == nullptr) return report(KVX_EINVAL, "cache is NULL");
  auto it = c->agents.find(agent);
  if (it == c->agents.end()) return report(KVX_EINVAL, "agent %lld is unknown", (long long)agent);
  if (it->second.active) return report(KVX_EINVAL, "agent %lld is inside a turn", (long long)agent);
  drop_tail(c, it->second, it->second.pages);
  drop_host(c, it->second, 0);
  if (it->second.in_group) {
    auto& m = c->groups[it->second.group].members;
    m.erase(std::find(m.begin(), m.end(), agent));
  }
  c->agents.erase(it);
  return KVX_OK;
}

int kvx_cache_agent(const kvx_cache* c, int64_t agent, int32_t* cached_tokens, int32_t* page_ids, int64_t cap) {
  if (c == nullptr || cached_tokens == nullptr) return report(KVX_EINVAL, "cache and cached_tokens must be non-NULL");
  auto it = c->agents.find(agent);
  if (it == c->agents.end()) {
    *cached_tokens = 0;
    return KVX_OK;
  }
  *cached_tokens = (int32_t)(it->second.pages * c->page_size);
  if (page_ids != nullptr) {
    int64_t j = 0;
    for (const CacheNode& nd : it->second.nodes)
      for (int32_t pg : nd.pages)
        if (j < cap) page_ids[j++] = pg;
  }
  return KVX_OK;
}

int kvx_cache_join(kvx_cache* c, int64_t agent, int64_t group, int32_t shared_tokens) {
  if (c == nullptr) return report(KVX_EINVAL, "cache is NULL");
  if (shared_tokens < c->page_size)
    return report(KVX_EINVAL, "shared_tokens = %d must cover at least one page", shared_tokens);
  const int64_t S = shared_tokens / c->page_size;
  auto ai = c->agents.find(agent);
  if (ai != c->agents.end()) {
    const CacheAgent& a = ai->second;
    if (a.active || a.pages > 0 || !a.host.empty() || a.in_group)
      return report(KVX_EINVAL, "agent %lld must be idle, hold no pages and belong to no group", (long long)agent);
  }
  auto gi = c->groups.find(group);
  if (gi != c->groups.end() && gi->second.S != S)
    return report(KVX_EINVAL, "group %lld shares %lld pages, not %lld", (long long)group, (long long)gi->second.S,
                  (long long)S);
  CacheGroup& g = c->groups[group];
  g.S = S;
  g.members.push_back(agent);
  CacheAgent& a = c->agents[agent];
  a.in_group = true;
  a.group = group;
  return KVX_OK;
}

int kvx_cache_group(const kvx_cache* c, int64_t group, int32_t* shared_tokens, int32_t* page_ids, int64_t cap) {
  if (c == nullptr || shared_tokens == nullptr) return report(KVX_EINVAL, "cache and shared_tokens must be non-NULL");
  auto it = c->groups.find(group);
  if (it == c->groups.end() || !it->second.present) {
    *shared_tokens = 0;
    return KVX_OK;
  }
  *shared_tokens = (int32_t)(it->second.S * c->page_size);
  if (page_ids != nullptr)
    for (int64_t j = 0; j < cap && j < (int64_t)it->second.pages.size(); j++) page_ids[j] = it->second.pages[(size_t)j];
  return KVX_OK;
}

int kvx_cache_agent_host(const kvx_cache* c, int64_t agent, int32_t* host_tokens, int32_t* slots, int64_t cap) {
  if (c == nullptr || host_tokens == nullptr) return report(KVX_EINVAL, "cache and host_tokens must be non-NULL");
  auto it = c->agents.find(agent);
  if (it == c->agents.end()) {
    *host_tokens = 0;
    return KVX_OK;
  }
  *host_tokens = (int32_t)((int64_t)it->second.host.size() * c->page_size);
  if (slots != nullptr) {
    int64_t j = 0;
    for (int32_t r : it->second.host)
      if (j < cap) slots[j++] = r;
  }
  return KVX_OK;
}

int kvx_cache_stats(const kvx_cache* c, kvx_cache_counters* out) {
  if (c == nullptr || out == nullptr) return report(KVX_EINVAL, "cache and out must be non-NULL");
  kvx_cache_counters s{};
  s.num_pages = c->num_pages;
  s.free_pages = (int64_t)c->free_pages.size();
  for (const auto& kv : c->agents) {
    s.cached_pages += kv.second.pages;
    s.turn_pages += (int64_t)kv.second.turn.size();
    if (kv.second.active) s.active_agents++;
  }
  s.agents = (int32_t)c->agents.size();
  s.evicted_pages = c->evicted_pages;
  s.evictions = c->evictions;
  s.host_pages = c->host_pages;
  s.host_used = c->host_used;
  s.spilled_pages = c->spilled;
  s.reloaded_pages = c->reloaded;
  s.host_dropped_pages = c->host_dropped;
  s.group_pages = c->group_pages;
  *out = s;
  return KVX_OK;
}

}  // extern "C"
