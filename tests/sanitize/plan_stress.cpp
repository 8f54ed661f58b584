// Host-only stress of the work planners (make_plan / make_decode_plan behind
// extend_attention_plan in csrc/kvx_host.cpp), built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_sanitizers.py.  The kernel launchers
// are replaced by stubs that must never run: planning touches no device.
//
// Seeded random ragged batches (empty and one-token suffixes, long prefixes, GQA
// groups from 1 to 32, forced and automatic splits) go through the plan, which must
// cover every (request, KV head, suffix token) by exactly one tile, partition each
// tile's key range [0, P + last token] at multiples of 64 (decode: into chunks of
// [0, P]), and number split parts densely.  Invalid batches must be refused.

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <tuple>
#include <vector>

#include "kvx_internal.h"

namespace kvx {
#define KVX_STUB(name, ...)                                       \
  hipError_t name(__VA_ARGS__) {                                  \
    std::fprintf(stderr, "planner stress: %s was called\n", #name); \
    std::exit(4);                                                 \
  }
KVX_STUB(launch_decode, const DecodeParams&, int64_t, int, bool, hipStream_t)
KVX_STUB(launch_decode_merge, const DecodeMergeParams&, int64_t, int, hipStream_t)
KVX_STUB(launch_extend_attention, const AttnParams&, int64_t, int, bool, bool, hipStream_t)
KVX_STUB(launch_merge, const MergeParams&, int64_t, int, hipStream_t)
KVX_STUB(launch_store_kv, const StoreParams&, int64_t, int, bool, hipStream_t)
KVX_STUB(launch_store_kv_rope, const RopeParams&, int64_t, int, bool, bool, hipStream_t)
KVX_STUB(launch_page_move, const PageMoveParams&, int64_t, hipStream_t)
KVX_STUB(launch_page_io, const PageIoParams&, int64_t, int, int, hipStream_t)
}  // namespace kvx

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      std::exit(3);                                                          \
    }                                                                        \
  } while (0)

namespace {

std::mt19937_64 rng(2024);
int64_t uni(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); }

void one(bool decode_like) {
  const int R = (int)uni(1, 12);
  const int hkv = (int)std::vector<int>{1, 2, 3, 8, 16}[(size_t)uni(0, 4)];
  const int g = (int)std::vector<int>{1, 2, 4, 8, 32}[(size_t)uni(0, 4)];
  const int D = uni(0, 1) ? 64 : 128;
  std::vector<int32_t> P((size_t)R), E((size_t)R), indptr((size_t)R + 1, 0);
  for (int r = 0; r < R; r++) {
    P[(size_t)r] = (int32_t)(uni(0, 3) == 0 ? 0 : uni(0, 200000));
    E[(size_t)r] = (int32_t)(decode_like ? uni(0, 1) : (uni(0, 4) == 0 ? 0 : uni(1, 3000)));
    indptr[(size_t)r + 1] = indptr[(size_t)r] + (P[(size_t)r] + E[(size_t)r] + 15) / 16 + (int32_t)uni(0, 2);
  }
  kvx_batch b{R, P.data(), E.data(), indptr.data(), nullptr};
  const int32_t splits[] = {0, 0, 64, 1024, 16384};
  const int32_t split = splits[uni(0, 4)];
  int64_t count = -1;
  CHECK(extend_attention_plan(&b, hkv * g, hkv, D, split, nullptr, 0, &count) == KVX_OK);
  std::vector<kvx_work_item> items((size_t)count + 1);
  int64_t count2 = -1;
  CHECK(extend_attention_plan(&b, hkv * g, hkv, D, split, items.data(), count, &count2) == KVX_OK);
  CHECK(count2 == count);
  items.resize((size_t)count);
  // (req, head, tok_begin) -> key ranges
  std::map<std::tuple<int, int, int>, std::vector<std::pair<int64_t, int64_t>>> cover;
  std::map<std::tuple<int, int, int>, int> tile_tokens;
  std::vector<int> part_seen;
  for (const kvx_work_item& it : items) {
    if (it.req < 0) continue;  // padding
    CHECK(it.req < R && it.kv_head >= 0 && it.kv_head < hkv);
    CHECK(it.key_begin >= 0 && it.key_begin < it.key_end);
    CHECK(it.tok_begin >= 0 && it.tok_count >= 1 && it.tok_begin + it.tok_count <= E[(size_t)it.req]);
    CHECK(it.key_end <= (int64_t)P[(size_t)it.req] + it.tok_begin + it.tok_count);
    CHECK(it.xcd >= 0 && it.xcd < 8);
    cover[{it.req, it.kv_head, it.tok_begin}].push_back({it.key_begin, it.key_end});
    auto tt = tile_tokens.emplace(std::make_tuple(it.req, it.kv_head, it.tok_begin), it.tok_count);
    CHECK(tt.first->second == it.tok_count);  // every part of a tile has the tile's tokens
    if (it.part >= 0) {
      if ((size_t)it.part >= part_seen.size()) part_seen.resize((size_t)it.part + 1, 0);
      part_seen[(size_t)it.part]++;
    }
  }
  for (int c : part_seen) CHECK(c == 1);  // parts numbered densely, each once
  for (int r = 0; r < R; r++) {
    for (int h = 0; h < hkv; h++) {
      int64_t tok = 0;
      while (tok < E[(size_t)r]) {
        auto f = cover.find({r, h, (int)tok});
        CHECK(f != cover.end());
        auto ranges = f->second;
        std::sort(ranges.begin(), ranges.end());
        CHECK(ranges.front().first == 0);
        for (size_t i = 1; i < ranges.size(); i++) {
          CHECK(ranges[i].first == ranges[i - 1].second);
          CHECK(ranges[i].first % 64 == 0);
        }
        const int ntok = tile_tokens[{r, h, (int)tok}];
        CHECK(ntok >= 1);
        CHECK(ranges.back().second == (int64_t)P[(size_t)r] + tok + ntok);
        cover.erase(f);
        tok += ntok;
      }
    }
  }
  CHECK(cover.empty());
}

}  // namespace

int main(int argc, char** argv) {
  const int n = argc > 1 ? std::atoi(argv[1]) : 300;
  for (int i = 0; i < n; i++) one(i % 4 == 3);
  // refused batches: negative lengths, too few pages, indptr not starting at 0
  int32_t P[1] = {-1}, E[1] = {4}, ip[2] = {0, 1};
  kvx_batch b{1, P, E, ip, nullptr};
  int64_t count = 0;
  CHECK(extend_attention_plan(&b, 4, 2, 128, 0, nullptr, 0, &count) == KVX_EINVAL);
  P[0] = 16;
  E[0] = 17;
  ip[1] = 2;
  CHECK(extend_attention_plan(&b, 4, 2, 128, 0, nullptr, 0, &count) == KVX_EINVAL);
  P[0] = 0;
  E[0] = 4;
  ip[0] = 1;
  ip[1] = 2;
  CHECK(extend_attention_plan(&b, 4, 2, 128, 0, nullptr, 0, &count) == KVX_EINVAL);
  CHECK(extend_attention_plan(&b, 4, 2, 128, 100, nullptr, 0, &count) == KVX_EINVAL);  // not a multiple of 64
  std::printf("planner stress: %d batches passed\n", n);
  return 0;
}
