// Host-only stress of the prefix cache (csrc/kvx_cache.cpp), built with
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_sanitizers.py.
//
// Seeded random turn sequences run for both policies, with and without a host
// tier, recency tiers and shared-prefix groups, through the C ABI of
// include/kvx_cache.h.  After every call the driver checks that every pool page
// is owned at most once (a group node, an agent's cached history, or the fresh
// pages of a running turn), that owned + free pages add up to the pool, that page
// ids and host records stay in range, and that no host record is held twice.
// Any failure, or any sanitizer report, ends the run with a nonzero status.

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <set>
#include <vector>

#include "kvx_cache.h"

// The library's error reporter (defined with the device code in the full build).
namespace kvx {
int report(int code, const char*, ...) { return code; }
}

namespace {

constexpr int kPage = 16;
int64_t g_nomem = 0, g_spills = 0, g_reloads = 0, g_evictions = 0, g_group_turns = 0;

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      std::exit(3);                                                          \
    }                                                                        \
  } while (0)

struct Run {
  kvx_cache* c = nullptr;
  int64_t num_pages = 0, host_pages = 0;
  std::map<int64_t, std::vector<int32_t>> tables;  // running turns
  std::set<int64_t> agents;                        // every agent ever started
  std::map<int64_t, int64_t> member;               // agent -> group
  std::set<int64_t> groups;

  std::vector<int32_t> agent_pages(int64_t a) const {
    int32_t tok = 0;
    CHECK(kvx_cache_agent(c, a, &tok, nullptr, 0) == KVX_OK);
    std::vector<int32_t> p((size_t)tok / kPage + 1);
    CHECK(kvx_cache_agent(c, a, &tok, p.data(), (int64_t)p.size()) == KVX_OK);
    p.resize((size_t)tok / kPage);
    return p;
  }
  std::vector<int32_t> group_pages(int64_t g) const {
    int32_t tok = 0;
    CHECK(kvx_cache_group(c, g, &tok, nullptr, 0) == KVX_OK);
    std::vector<int32_t> p((size_t)tok / kPage + 1);
    CHECK(kvx_cache_group(c, g, &tok, p.data(), (int64_t)p.size()) == KVX_OK);
    p.resize((size_t)tok / kPage);
    return p;
  }

  void check() const {
    kvx_cache_counters st{};
    CHECK(kvx_cache_stats(c, &st) == KVX_OK);
    std::vector<int32_t> owned;
    int64_t gp = 0;
    for (int64_t g : groups) {
      auto p = group_pages(g);
      gp += (int64_t)p.size();
      owned.insert(owned.end(), p.begin(), p.end());
    }
    CHECK(gp == st.group_pages);
    std::set<int32_t> host_slots;
    int64_t host_held = 0;
    for (int64_t a : agents) {
      auto p = agent_pages(a);
      owned.insert(owned.end(), p.begin(), p.end());
      int32_t htok = 0;
      CHECK(kvx_cache_agent_host(c, a, &htok, nullptr, 0) == KVX_OK);
      std::vector<int32_t> s((size_t)htok / kPage + 1);
      CHECK(kvx_cache_agent_host(c, a, &htok, s.data(), (int64_t)s.size()) == KVX_OK);
      for (int i = 0; i < htok / kPage; i++) {
        CHECK(s[(size_t)i] >= 0 && s[(size_t)i] < host_pages);
        CHECK(host_slots.insert(s[(size_t)i]).second);
        host_held++;
      }
    }
    CHECK(host_held == st.host_used);
    for (const auto& kv : tables) {
      std::set<int32_t> skip;
      auto it = member.find(kv.first);
      if (it != member.end())
        for (int32_t p : group_pages(it->second)) skip.insert(p);
      for (int32_t p : agent_pages(kv.first)) skip.insert(p);
      for (int32_t p : kv.second)
        if (!skip.count(p)) owned.push_back(p);
    }
    std::set<int32_t> uniq(owned.begin(), owned.end());
    CHECK(uniq.size() == owned.size());
    for (int32_t p : owned) CHECK(p >= 0 && p < num_pages);
    CHECK((int64_t)owned.size() + st.free_pages == num_pages);
  }
};

// One trace: `steps` random actions over `n_agents` agents.
void trace(uint64_t seed, int policy, int64_t num_pages, int64_t host_pages, int chunk_tokens, int64_t tiers,
           bool with_groups, int steps) {
  std::mt19937_64 rng(seed);
  auto uni = [&](int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); };
  Run r;
  r.num_pages = num_pages;
  r.host_pages = host_pages;
  CHECK(kvx_cache_create_tiered(num_pages, host_pages, kPage, chunk_tokens, policy, &r.c) == KVX_OK);
  if (tiers > 0) CHECK(kvx_cache_set_recency_tiers(r.c, tiers) == KVX_OK);
  const int n_agents = 12;
  std::map<int64_t, int32_t> ctx;  // agent -> context length so far
  std::vector<int32_t> table((size_t)num_pages + 64);
  for (int step = 0; step < steps; step++) {
    const int64_t a = uni(0, n_agents - 1);
    const bool active = r.tables.count(a) != 0;
    const int action = (int)uni(0, 99);
    if (active) {
      if (action < 80) {
        CHECK(kvx_cache_end_turn(r.c, a) == KVX_OK);
        r.tables.erase(a);
      } else {
        // an illegal call on an active agent leaves everything as it was
        int32_t pre = 0;
        kvx_cache_moves mv{};
        CHECK(kvx_cache_begin_turn_tiered(r.c, a, 100, &pre, table.data(), (int64_t)table.size(), &mv) ==
              KVX_EINVAL);
        CHECK(kvx_cache_complete(r.c, a) == KVX_EINVAL);
      }
    } else if (action < 6 && r.agents.count(a)) {
      CHECK(kvx_cache_complete(r.c, a) == KVX_OK);
      r.agents.erase(a);
      r.member.erase(a);
      ctx.erase(a);
    } else {
      if (with_groups && !r.agents.count(a) && action % 3 == 0) {
        const int64_t g = a % 2;
        const int32_t shared = g == 0 ? 6 * kPage : 3 * kPage;
        CHECK(kvx_cache_join(r.c, a, g, shared + (int32_t)uni(0, kPage - 1)) == KVX_OK);
        r.member[a] = g;
        r.groups.insert(g);
      }
      const int32_t grow = (int32_t)uni(1, 8 * kPage);
      int32_t len = ctx.count(a) ? ctx[a] + grow : grow + (int32_t)uni(0, 6 * kPage);
      if (len > (int32_t)(num_pages * kPage / 3)) len = (int32_t)uni(1, 4 * kPage);  // a fresh task
      auto mem = r.member.find(a);
      if (mem != r.member.end()) {  // a member's context starts with the group's shared pages
        const int32_t span = mem->second == 0 ? 6 * kPage : 3 * kPage;
        if (len <= span) len = span + (int32_t)uni(1, 2 * kPage);
      }
      int32_t pre = -1;
      kvx_cache_moves mv{};
      const int rc = kvx_cache_begin_turn_tiered(r.c, a, len, &pre, table.data(), (int64_t)table.size(), &mv);
      CHECK(rc == KVX_OK || rc == KVX_ENOMEM);
      g_nomem += rc == KVX_ENOMEM;
      g_spills += mv.n_spill;
      g_group_turns += rc == KVX_OK && mem != r.member.end();
      for (int64_t i = 0; i < mv.n_spill; i++) {
        CHECK(mv.spill_pages[i] >= 0 && mv.spill_pages[i] < num_pages);
        CHECK(mv.spill_slots[i] >= 0 && mv.spill_slots[i] < host_pages);
      }
      r.agents.insert(a);
      if (rc == KVX_OK) {
        CHECK(pre >= 0 && pre < len && pre % kPage == 0);
        g_reloads += mv.n_reload;
        for (int64_t i = 0; i < mv.n_reload; i++) {
          CHECK(mv.reload_pages[i] >= 0 && mv.reload_pages[i] < num_pages);
          CHECK(mv.reload_slots[i] >= 0 && mv.reload_slots[i] < host_pages);
        }
        const int n = (len + kPage - 1) / kPage;
        r.tables[a] = std::vector<int32_t>(table.begin(), table.begin() + n);
        ctx[a] = len;
      }
    }
    r.check();
  }
  for (auto it = r.tables.begin(); it != r.tables.end(); it = r.tables.erase(it))
    CHECK(kvx_cache_end_turn(r.c, it->first) == KVX_OK);
  r.check();
  kvx_cache_counters st{};
  CHECK(kvx_cache_stats(r.c, &st) == KVX_OK);
  g_evictions += st.evictions;
  CHECK(kvx_cache_destroy(r.c) == KVX_OK);
}

}  // namespace

int main(int argc, char** argv) {
  const int steps = argc > 1 ? std::atoi(argv[1]) : 400;
  int n = 0;
  for (int policy : {KVX_EVICT_LRU, KVX_EVICT_RR})
    for (int64_t host : {0, 24})
      for (bool groups : {false, true})
        for (int64_t tiers : {0, 7}) {
          if (tiers && policy != KVX_EVICT_RR) continue;
          for (uint64_t seed = 1; seed <= 3; seed++) {
            trace(seed * 1000 + (uint64_t)n, policy, 96, host, 2 * kPage, tiers, groups, steps);
            n++;
          }
        }
  // degenerate pools: a single page, and chunks longer than any history
  trace(7, KVX_EVICT_RR, 1, 0, kPage, 0, false, steps / 4);
  trace(8, KVX_EVICT_LRU, 1, 2, kPage, 0, false, steps / 4);
  trace(9, KVX_EVICT_RR, 40, 8, 64 * kPage, 3, true, steps);
  std::printf("cache stress: %d traces of %d steps passed (%lld evictions, %lld ENOMEM turn starts, "
              "%lld spills, %lld reloads, %lld group-member turns)\n",
              n + 3, steps, (long long)g_evictions, (long long)g_nomem, (long long)g_spills, (long long)g_reloads,
              (long long)g_group_turns);
  return 0;
}
