// Host-only stress of the token-content prefix cache (csrc/kvx_radix.cpp), built
// with AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_sanitizers.py.
//
// Seeded random request sequences of agents that share a prompt, extend their
// histories, retry from earlier points and fork each other's histories run for
// both policies through the C ABI of include/kvx_radix.h.  After every call the
// driver checks that free + cached + temporary pages add up to the pool, that
// every page table holds distinct in-range pages whose reused part is the tree's
// match, and that a finished request's whole pages are found by the match probe.
// Any failure, or any sanitizer report, ends the run with a nonzero status.

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <set>
#include <vector>

#include "kvx_cache.h"
#include "kvx_radix.h"

// The library's error reporter (defined with the device code in the full build).
namespace kvx {
int report(int code, const char*, ...) { return code; }
}

namespace {

constexpr int kPage = 16;
int64_t g_nomem = 0, g_reused = 0;

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      std::exit(3);                                                          \
    }                                                                        \
  } while (0)

void one(uint32_t seed, int policy) {
  std::mt19937 rng(seed);
  auto uni = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  const int64_t num_pages = uni(20, 200);
  kvx_radix* t = nullptr;
  CHECK(kvx_radix_create(num_pages, kPage, kPage * uni(1, 4), policy, &t) == KVX_OK);
  const int agents = uni(2, 8);
  std::vector<int32_t> system((size_t)uni(0, 60));
  for (auto& x : system) x = uni(0, 7);
  std::vector<std::vector<int32_t>> hist((size_t)agents, system);
  std::set<int> running;
  for (int step = 0; step < 300; step++) {
    const int a = uni(0, agents - 1);
    if (running.count(a)) {
      CHECK(kvx_radix_end(t, a) == KVX_OK);
      running.erase(a);
    } else {
      const int u = uni(0, 99);
      auto& h = hist[(size_t)a];
      if (u < 10 && !h.empty()) h.resize((size_t)uni(0, (int)h.size()));
      if (u >= 10 && u < 15) h = hist[(size_t)uni(0, agents - 1)];
      if (u >= 15 && u < 18) {
        CHECK(kvx_radix_complete(t, a) == KVX_OK);
        continue;
      }
      const int add = uni(1, 100);
      for (int i = 0; i < add; i++) h.push_back(uni(0, 7));  // few symbols: many shared pages
      const int n = (int)h.size();
      std::vector<int32_t> table((size_t)((n + kPage - 1) / kPage) + 1, -7);
      int32_t prefix = -1, matched = -1;
      CHECK(kvx_radix_match(t, h.data(), n, &matched, nullptr, 0) == KVX_OK);
      const int rc = kvx_radix_begin(t, a, h.data(), n, &prefix, table.data(), (int64_t)table.size());
      if (rc == KVX_ENOMEM) {
        g_nomem++;
      } else {
        CHECK(rc == KVX_OK);
        running.insert(a);
        const int np = (n + kPage - 1) / kPage;
        CHECK(prefix % kPage == 0 && prefix <= n - 1 && prefix <= matched);
        CHECK(table[(size_t)np] == -7);  // nothing written past the table
        std::set<int32_t> seen;
        for (int i = 0; i < np; i++) {
          CHECK(table[(size_t)i] >= 0 && table[(size_t)i] < num_pages);
          CHECK(seen.insert(table[(size_t)i]).second);
        }
        std::vector<int32_t> mp((size_t)(n / kPage) + 1);
        int32_t m2 = 0;
        CHECK(kvx_radix_match(t, h.data(), n, &m2, mp.data(), (int64_t)mp.size()) == KVX_OK);
        CHECK(m2 == (n / kPage) * kPage);  // the prompt's whole pages are in the tree now
        for (int i = 0; i < prefix / kPage; i++) CHECK(mp[(size_t)i] == table[(size_t)i]);
        g_reused += prefix > 0;
      }
    }
    kvx_radix_counters c{};
    CHECK(kvx_radix_stats(t, &c) == KVX_OK);
    CHECK(c.free_pages + c.cached_pages + c.temp_pages == num_pages);
    CHECK(c.active == (int32_t)running.size());
    CHECK(c.leaves <= c.nodes);
  }
  CHECK(kvx_radix_destroy(t) == KVX_OK);
}

}  // namespace

int main(int argc, char** argv) {
  const int n = argc > 1 ? std::atoi(argv[1]) : 200;
  for (int i = 0; i < n; i++) one((uint32_t)i, i % 2 ? KVX_EVICT_RR : KVX_EVICT_LRU);
  CHECK(g_reused > 0 && g_nomem > 0);
  std::printf("radix stress: %d runs passed (%lld requests reused a prefix, %lld refused)\n", n, (long long)g_reused,
              (long long)g_nomem);
  return 0;
}
