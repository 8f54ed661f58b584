// Host side of libkvx: the C ABI declared in include/kvx.h.
//
// Owns the KV pool (hipMalloc), checks every argument before queuing work,
// plans extend_attention's work over ragged (prefix_len, extend_len) pairs and
// uploads the plan through pinned staging buffers on the caller's stream.

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <numeric>
#include <string>
#include <tuple>
#include <vector>

#include "kvx_internal.h"

using kvx::AttnUnit;
using kvx::MergeUnit;
using kvx::StoreUnit;

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

}  // namespace

int kvx::report(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? KVX_ENOMEM : KVX_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define KVX_HIP(call)                                   \
  do {                                                  \
    hipError_t e_ = (call);                             \
    if (e_ != hipSuccess) return hip_fail(e_, #call);   \
  } while (0)

bool validate_mode() {
  const char* v = std::getenv("KVX_VALIDATE");
  return v != nullptr && v[0] != '\0' && v[0] != '0';
}

// Pinned host buffer + device buffer + events: a reusable upload channel.  The
// host side is rewritten only after the previous copy out of it has completed.
// The device buffer grows with the stream-ordered allocator: the old buffer is
// freed in stream order behind `used` (recorded after the last kernels that read
// it), so growing never waits on the host for the device.
struct Staging {
  void* host = nullptr;
  size_t host_cap = 0;
  void* dev = nullptr;
  size_t dev_cap = 0;
  hipEvent_t ev = nullptr;    // after the last copy out of `host`
  hipEvent_t used = nullptr;  // after the last kernels that read `dev`
  bool pending = false;

  // Only after the device has gone idle (pool destruction).
  void release() {
    if (ev) {
      (void)hipEventSynchronize(ev);
      (void)hipEventDestroy(ev);
    }
    if (used) (void)hipEventDestroy(used);
    if (host) (void)hipHostFree(host);
    if (dev) (void)hipFreeAsync(dev, nullptr);
    *this = Staging();
  }

  // Copy `bytes` from `src` to device memory ordered on `stream`; *out receives the
  // device address (valid until the next upload on this channel is ordered after it).
  // The caller records done() on the stream after the kernels that read it.
  int upload(const void* src, size_t bytes, hipStream_t stream, void** out) {
    if (!ev) KVX_HIP(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
    if (!used) KVX_HIP(hipEventCreateWithFlags(&used, hipEventDisableTiming));
    if (pending) {
      KVX_HIP(hipEventSynchronize(ev));
      pending = false;
    }
    if (bytes > host_cap) {
      if (host) KVX_HIP(hipHostFree(host));
      host = nullptr;
      size_t cap = std::max<size_t>(bytes + bytes / 2, 4096);
      KVX_HIP(hipHostMalloc(&host, cap, hipHostMallocDefault));
      host_cap = cap;
    }
    if (bytes > dev_cap) {
      if (dev) {
        // earlier kernels (on any stream) that read the old buffer precede `used`
        KVX_HIP(hipStreamWaitEvent(stream, used, 0));
        KVX_HIP(hipFreeAsync(dev, stream));
      }
      dev = nullptr;
      dev_cap = 0;
      size_t cap = std::max<size_t>(bytes + bytes / 2, 4096);
      KVX_HIP(hipMallocAsync(&dev, cap, stream));
      dev_cap = cap;
    }
    std::memcpy(host, src, bytes);
    KVX_HIP(hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, stream));
    KVX_HIP(hipEventRecord(ev, stream));
    pending = true;
    *out = dev;
    return KVX_OK;
  }

  int done(hipStream_t stream) {
    KVX_HIP(hipEventRecord(used, stream));
    return KVX_OK;
  }
};

// Device scratch that only grows, with the same stream-ordered replacement.
struct Workspace {
  void* ptr = nullptr;
  size_t cap = 0;
  hipEvent_t used = nullptr;  // after the last kernels that used `ptr`
  int ensure(size_t bytes, hipStream_t stream) {
    if (!used) KVX_HIP(hipEventCreateWithFlags(&used, hipEventDisableTiming));
    if (bytes <= cap) return KVX_OK;
    if (ptr) {
      KVX_HIP(hipStreamWaitEvent(stream, used, 0));
      KVX_HIP(hipFreeAsync(ptr, stream));
      ptr = nullptr;
      cap = 0;
    }
    // headroom of a quarter for small sizes; past 1 GiB exactly what is asked
    size_t c = bytes > ((size_t)1 << 30) ? bytes : std::max<size_t>(bytes + bytes / 4, 1 << 20);
    KVX_HIP(hipMallocAsync(&ptr, c, stream));
    cap = c;
    return KVX_OK;
  }
  int done(hipStream_t stream) {
    if (used) KVX_HIP(hipEventRecord(used, stream));
    return KVX_OK;
  }
  // Only after the device has gone idle (pool destruction).
  void release() {
    if (ptr) (void)hipFreeAsync(ptr, nullptr);
    if (used) (void)hipEventDestroy(used);
    ptr = nullptr;
    cap = 0;
    used = nullptr;
  }
};

constexpr int kPlanSlots = 256;  // 256 CUs x 1 resident attention workgroup
// Bound on the partial results of split key ranges: 16384 parts x 256 rows x 128
// dims x 4 B = 2 GiB (+16 MiB of LSE) at head_dim 128, allocated exactly.
constexpr int64_t kMaxParts = 16384;

}  // namespace

struct kvx_pool {
  int device = 0;
  int64_t num_pages = 0;
  int32_t page_size = 16;
  int32_t num_kv_heads = 0;
  int32_t head_dim = 0;
  int32_t kv_dtype = KVX_KV_BF16;
  int32_t elem_bytes = 2;
  void* k = nullptr;
  void* v = nullptr;
  float* scales_d = nullptr;  // [k_scale | v_scale | k_inv | v_inv], each num_kv_heads
  Staging st_store, st_attn, st_io, st_move;
  Workspace parts;
  int32_t split_keys = 0;  // key-range split length of extend_attention; 0 = automatic
  int32_t scaled_q = 0;    // 1: prefill attention on a bf16 pool takes the folded softmax
};

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int check_pool(const kvx_pool* pool) {
  if (pool == nullptr) return fail(KVX_EINVAL, "pool is NULL");
  return KVX_OK;
}

// The kernels move 16-byte pieces: every bf16 row buffer must start 16-byte aligned.
int check_align(const void* ptr, const char* name) {
  if (ptr != nullptr && ((uintptr_t)ptr & 15u) != 0)
    return fail(KVX_EINVAL, "%s = %p is not 16-byte aligned", name, ptr);
  return KVX_OK;
}

int use_device(const kvx_pool* pool) {
  int cur = -1;
  KVX_HIP(hipGetDevice(&cur));
  if (cur != pool->device) KVX_HIP(hipSetDevice(pool->device));
  return KVX_OK;
}

// Host-side checks of a batch; fills qo offsets (request r owns rows [qo[r], qo[r+1])).
int check_batch(const kvx_batch* b, std::vector<int64_t>& qo, bool need_page_ids = true) {
  if (b == nullptr) return fail(KVX_EINVAL, "batch is NULL");
  if (b->num_reqs < 0) return fail(KVX_EINVAL, "num_reqs = %d < 0", b->num_reqs);
  qo.assign((size_t)b->num_reqs + 1, 0);
  if (b->num_reqs == 0) return KVX_OK;
  if (!b->prefix_lens || !b->extend_lens || !b->page_indptr)
    return fail(KVX_EINVAL, "prefix_lens, extend_lens and page_indptr must be non-NULL");
  if (b->page_indptr[0] != 0) return fail(KVX_EINVAL, "page_indptr[0] = %d, must be 0", b->page_indptr[0]);
  for (int r = 0; r < b->num_reqs; r++) {
    const int64_t P = b->prefix_lens[r], E = b->extend_lens[r];
    if (P < 0 || E < 0) return fail(KVX_EINVAL, "request %d: negative length (P=%lld, E=%lld)", r, (long long)P, (long long)E);
    if (P + E > (int64_t)INT32_MAX - 1024) return fail(KVX_EINVAL, "request %d: sequence too long", r);
    const int64_t have = (int64_t)b->page_indptr[r + 1] - b->page_indptr[r];
    if (have < ceil_div(P + E, kvx::kPageSize))
      return fail(KVX_EINVAL, "request %d: %lld page ids for %lld tokens (need %lld)", r, (long long)have,
                  (long long)(P + E), (long long)ceil_div(P + E, kvx::kPageSize));
    qo[r + 1] = qo[r] + E;
  }
  if (qo.back() > (int64_t)INT32_MAX) return fail(KVX_EINVAL, "total extend length exceeds 2^31-1");
  if (need_page_ids && b->page_indptr[b->num_reqs] > 0 && b->page_ids == nullptr)
    return fail(KVX_EINVAL, "page_ids is NULL");
  return KVX_OK;
}

// KVX_VALIDATE=1: copy the page table to the host and check every id.
int check_page_ids(const kvx_pool* pool, const kvx_batch* b, hipStream_t stream) {
  const int64_t n = b->num_reqs ? b->page_indptr[b->num_reqs] : 0;
  if (n == 0) return KVX_OK;
  std::vector<int32_t> ids((size_t)n);
  KVX_HIP(hipStreamSynchronize(stream));
  KVX_HIP(hipMemcpy(ids.data(), b->page_ids, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost));
  for (int64_t i = 0; i < n; i++)
    if (ids[(size_t)i] < 0 || ids[(size_t)i] >= pool->num_pages)
      return fail(KVX_ERANGE, "page_ids[%lld] = %d outside [0, %lld)", (long long)i, ids[(size_t)i],
                  (long long)pool->num_pages);
  return KVX_OK;
}

struct Plan {
  std::vector<AttnUnit> units;  // in launch order (position i runs on XCD i % 8)
  std::vector<MergeUnit> merges;
  std::vector<kvx_work_item> items;  // same order, for inspection
  int64_t n_parts = 0;
};

// Work plan of extend_attention.
//   * every request's suffix is cut into tiles of tile_tok tokens (x group query heads
//     = 256 rows) per KV head; a tile covers keys [0, P + last token of the tile];
//   * when the batch has too little work to fill the chip, or a tile's key range is
//     far longer than the average work per workgroup slot, the key range is split at
//     multiples of the tile width into parts merged by log-sum-exp afterwards (the
//     parts lengthened slightly when that saves a nearly empty last round of units);
//   * each (request, KV head) is bound to one XCD (KV head h -> XCD h % 8 when the
//     head count is a multiple of 8), so the workgroups that stream the same K/V
//     pages share one L2; for other head counts each (request, KV head, part of a
//     split key range) is bound greedily by cost, so that a batch of few long
//     requests still spreads its parts over all eight XCDs (the parts of one key
//     range, read by every tile of the request, stay together);
//   * within an XCD, requests go longest first and a request's tiles longest first.
int make_plan(const kvx_batch* b, const std::vector<int64_t>& qo, int32_t Hq, int32_t Hkv, int32_t split_keys,
              int64_t max_parts, Plan& plan) {
  const int G = Hq / Hkv;
  const int tile_tok = kvx::kTileRows / G;
  const int BN = kvx::kTileKeys;

  struct Tile { int r, h, tok0, ntok; int64_t kend, qpos0, cost; };
  std::vector<Tile> tiles;
  int64_t total_cost = 0, max_cost = 0;
  for (int r = 0; r < b->num_reqs; r++) {
    const int64_t P = b->prefix_lens[r], E = b->extend_lens[r];
    for (int64_t t0 = 0; t0 < E; t0 += tile_tok) {
      const int ntok = (int)std::min<int64_t>(tile_tok, E - t0);
      const int64_t kend = P + t0 + ntok;
      const int64_t cost = ceil_div(kend, BN);
      for (int h = 0; h < Hkv; h++) {
        tiles.push_back(Tile{r, h, (int)t0, ntok, kend, P + t0, cost});
        total_cost += cost;
        max_cost = std::max(max_cost, cost);
      }
    }
  }

  // split length in keys (a multiple of BN), 0 = no split
  int64_t split = 0;
  if (split_keys > 0) {
    split = split_keys;
  } else if (!tiles.empty()) {
    const int64_t avg = total_cost / kPlanSlots;            // tiles of keys per slot
    const int64_t allowed = std::max<int64_t>(avg / 2, 16);  // at least 1024 keys per part
    if (max_cost > allowed) split = allowed * BN;
  }
  if (split > 0) {
    // keep the number of parts bounded
    for (;;) {
      int64_t parts = 0;
      for (const Tile& t : tiles) {
        const int64_t nb = t.qpos0 / split;  // boundaries split, 2 split, ... <= qpos0
        if (nb > 0) parts += nb + 1;
      }
      if (parts <= max_parts) break;
      split *= 2;
    }
    if (split_keys <= 0) {
      // Whole rounds: a unit count a little past a multiple of the 256 slots leaves a
      // nearly empty last round.  Lengthen the parts (in whole tiles) when that
      // removes it for less than half a round (the units spilling into it are often
      // a tile's short last parts): the smallest split below split * (1 + 1 / 2k)
      // that yields at most k rounds of units (the count never grows with the
      // split, so a bisection finds it).
      std::vector<std::pair<int64_t, int64_t>> starts;  // (first query position, tiles)
      for (const Tile& t : tiles) {
        if (!starts.empty() && starts.back().first == t.qpos0) starts.back().second++;
        else starts.push_back({t.qpos0, 1});
      }
      auto units_at = [&](int64_t s) {
        int64_t n = 0;
        for (const auto& q : starts) n += (q.first / s + 1) * q.second;
        return n;
      };
      const int64_t k = (units_at(split) - 1) / kPlanSlots;
      if (k >= 1) {
        const int64_t target = k * kPlanSlots;
        int64_t lo = split / BN + 1, hi = (split + split / (2 * k) - 1) / BN;  // split lengths in tiles
        if (lo <= hi && units_at(hi * BN) <= target) {
          while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            if (units_at(mid * BN) <= target) hi = mid;
            else lo = mid + 1;
          }
          split = lo * BN;
        }
      }
    }
  }

  // Key ranges of a tile: [0, split), [split, 2 split), ... up to the last boundary
  // <= qpos0, then the rest to kend; one range when unsplit.
  auto ranges_of = [&](const Tile& t) {
    std::vector<std::pair<int64_t, int64_t>> rg;
    if (split > 0 && t.qpos0 / split > 0) {
      int64_t kb = 0;
      for (int64_t bnd = split; bnd <= t.qpos0; bnd += split) {
        rg.push_back({kb, bnd});
        kb = bnd;
      }
      rg.push_back({kb, t.kend});
    } else {
      rg.push_back({0, t.kend});
    }
    return rg;
  };
  // XCD of (request, head, part index).  Multiples of 8 heads: head h -> XCD h % 8
  // for every part.  Otherwise greedy by cost over (request, head, part) keys,
  // costliest first, each to the least loaded XCD.
  const bool by_head = Hkv % kvx::kNumXcd == 0;
  std::map<std::tuple<int, int, int64_t>, int> bind_xcd;
  if (!by_head) {
    std::map<std::tuple<int, int, int64_t>, int64_t> bind_cost;
    for (const Tile& t : tiles) {
      const auto rg = ranges_of(t);
      for (size_t i = 0; i < rg.size(); i++)
        bind_cost[{t.r, t.h, (int64_t)i}] += ceil_div(rg[i].second - rg[i].first, BN);
    }
    std::vector<std::pair<std::tuple<int, int, int64_t>, int64_t>> order(bind_cost.begin(), bind_cost.end());
    std::stable_sort(order.begin(), order.end(), [](const auto& a, const auto& c) { return a.second > c.second; });
    int64_t load[kvx::kNumXcd] = {0};
    for (const auto& kc : order) {
      int best = 0;
      for (int x = 1; x < kvx::kNumXcd; x++)
        if (load[x] < load[best]) best = x;
      bind_xcd[kc.first] = best;
      load[best] += kc.second;
    }
  }
  // request order: total cost, longest first
  std::vector<int64_t> req_cost((size_t)b->num_reqs, 0);
  for (const Tile& t : tiles) req_cost[(size_t)t.r] += t.cost;
  std::vector<int> req_rank((size_t)b->num_reqs);
  {
    std::vector<int> order((size_t)b->num_reqs);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int a, int c) { return req_cost[(size_t)a] > req_cost[(size_t)c]; });
    for (int i = 0; i < b->num_reqs; i++) req_rank[(size_t)order[(size_t)i]] = i;
  }
  std::stable_sort(tiles.begin(), tiles.end(), [&](const Tile& a, const Tile& c) {
    if (req_rank[(size_t)a.r] != req_rank[(size_t)c.r]) return req_rank[(size_t)a.r] < req_rank[(size_t)c.r];
    if (a.cost != c.cost) return a.cost > c.cost;
    return a.h < c.h;
  });

  std::vector<std::vector<AttnUnit>> per_xcd(kvx::kNumXcd);
  std::vector<std::vector<kvx_work_item>> per_xcd_items(kvx::kNumXcd);
  plan.merges.clear();
  plan.n_parts = 0;
  for (const Tile& t : tiles) {
    AttnUnit u;
    u.qo_row0 = (int32_t)(qo[(size_t)t.r] + t.tok0);
    u.q_pos0 = (int32_t)t.qpos0;
    u.page_base = b->page_indptr[t.r];
    u.head_ntok = (t.h << 16) | t.ntok;
    u.req = t.r;
    const std::vector<std::pair<int64_t, int64_t>> ranges = ranges_of(t);
    const bool is_split = ranges.size() > 1;
    if (is_split) {
      MergeUnit m;
      m.qo_row0 = u.qo_row0;
      m.head_ntok = u.head_ntok;
      m.part0 = (int32_t)plan.n_parts;
      m.nparts = (int32_t)ranges.size();
      plan.merges.push_back(m);
    }
    for (size_t i = 0; i < ranges.size(); i++) {
      const auto& rg = ranges[i];
      const int x = by_head ? t.h % kvx::kNumXcd : bind_xcd.at({t.r, t.h, (int64_t)i});
      u.key_begin = (int32_t)rg.first;
      u.key_end = (int32_t)rg.second;
      u.part = is_split ? (int32_t)plan.n_parts++ : -1;
      per_xcd[(size_t)x].push_back(u);
      per_xcd_items[(size_t)x].push_back(kvx_work_item{t.r, t.h, t.tok0, t.ntok, u.key_begin, u.key_end, u.part, x});
    }
  }
  size_t longest = 0;
  for (const auto& v : per_xcd) longest = std::max(longest, v.size());
  plan.units.clear();
  plan.items.clear();
  for (size_t i = 0; i < longest; i++) {
    for (int x = 0; x < kvx::kNumXcd; x++) {
      if (i < per_xcd[(size_t)x].size()) {
        plan.units.push_back(per_xcd[(size_t)x][i]);
        plan.items.push_back(per_xcd_items[(size_t)x][i]);
      } else {
        AttnUnit pad{};
        pad.key_begin = 0;
        pad.key_end = 0;
        pad.part = -1;
        plan.units.push_back(pad);
        plan.items.push_back(kvx_work_item{-1, 0, 0, 0, 0, 0, -1, x});
      }
    }
  }
  // drop trailing padding
  while (!plan.units.empty() && plan.units.back().key_end <= plan.units.back().key_begin) {
    plan.units.pop_back();
    plan.items.pop_back();
  }
  return KVX_OK;
}

// ---- decode steps: every request with work has exactly one suffix token
using kvx::DecodeMerge;
using kvx::DecodeUnit;

struct DecodePlan {
  std::vector<DecodeUnit> units;
  std::vector<DecodeMerge> merges;
  std::vector<kvx_work_item> items;
  int64_t n_parts = 0;
};

bool is_decode_batch(const kvx_batch* b, int32_t Hq, int32_t Hkv) {
  if (Hq / Hkv > kvx::kDecodeMaxGroup) return false;
  bool any = false;
  for (int r = 0; r < b->num_reqs; r++) {
    if (b->extend_lens[r] > 1) return false;
    any |= b->extend_lens[r] == 1;
  }
  return any;
}

// Work plan of a decode step: each (request, KV head) key range [0, P] is cut into
// chunks of a common length, a multiple of 64 keys chosen so that the batch yields
// about 2048 chunks (8 per workgroup slot at two resident workgroups per CU), at
// least 512 keys each; a range of more than one chunk becomes parts merged by
// log-sum-exp.  Chunks are dispatched longest first.
int make_decode_plan(const kvx_batch* b, const std::vector<int64_t>& qo, int32_t Hkv, int32_t split_keys,
                     int64_t max_parts, DecodePlan& plan) {
  const int64_t A = kvx::kDecodeChunkAlign;
  int64_t total = 0;
  for (int r = 0; r < b->num_reqs; r++)
    if (b->extend_lens[r] == 1) total += (int64_t)Hkv * ((int64_t)b->prefix_lens[r] + 1);
  int64_t chunk;
  if (split_keys > 0) {
    chunk = split_keys;
  } else {
    chunk = std::max<int64_t>(512, (total + 2047) / 2048);
    chunk = (chunk + A - 1) / A * A;
  }
  for (;;) {  // bound the partial results like the prefill planner does
    int64_t parts = 0;
    for (int r = 0; r < b->num_reqs; r++) {
      if (b->extend_lens[r] != 1) continue;
      const int64_t n = ((int64_t)b->prefix_lens[r] + 1 + chunk - 1) / chunk;
      if (n > 1) parts += n * Hkv;
    }
    if (parts <= max_parts) break;
    chunk *= 2;
  }
  for (int r = 0; r < b->num_reqs; r++) {
    if (b->extend_lens[r] != 1) continue;
    const int64_t L = (int64_t)b->prefix_lens[r] + 1;
    const int64_t nc = (L + chunk - 1) / chunk;
    for (int32_t h = 0; h < Hkv; h++) {
      const int64_t part0 = plan.n_parts;
      for (int64_t c = 0; c < nc; c++) {
        DecodeUnit u{};
        u.qo_row = (int32_t)qo[(size_t)r];
        u.page_base = b->page_indptr[r];
        u.key_begin = (int32_t)(c * chunk);
        u.key_end = (int32_t)std::min<int64_t>(L, (c + 1) * chunk);
        u.head = h;
        u.part = nc > 1 ? (int32_t)plan.n_parts++ : -1;
        u.req = r;
        plan.units.push_back(u);
      }
      if (nc > 1) plan.merges.push_back(DecodeMerge{(int32_t)qo[(size_t)r], h, (int32_t)part0, (int32_t)nc});
    }
  }
  std::stable_sort(plan.units.begin(), plan.units.end(), [](const DecodeUnit& x, const DecodeUnit& y) {
    return x.key_end - x.key_begin > y.key_end - y.key_begin;
  });
  for (size_t i = 0; i < plan.units.size(); i++) {
    const DecodeUnit& u = plan.units[i];
    kvx_work_item it{u.req, u.head, 0, 1, u.key_begin, u.key_end, u.part, (int32_t)(i % kvx::kNumXcd)};
    plan.items.push_back(it);
  }
  return KVX_OK;
}

int check_heads(int32_t Hq, int32_t Hkv, int32_t D) {
  if (Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0)
    return fail(KVX_EINVAL, "num_q_heads (%d) must be a positive multiple of num_kv_heads (%d)", Hq, Hkv);
  if (Hq / Hkv > kvx::kTileRows)
    return fail(KVX_EUNSUPPORTED, "query heads per KV head (%d) above %d", Hq / Hkv, kvx::kTileRows);
  if (Hkv >= (1 << 15)) return fail(KVX_EUNSUPPORTED, "num_kv_heads too large");
  if (D != 64 && D != 128) return fail(KVX_EUNSUPPORTED, "head_dim %d (supported: 64, 128)", D);
  return KVX_OK;
}

// Where one attention call keeps its plan and its partial results: the pool's
// growable buffers, or the caller-independent fixed scratch of the allocation-free
// entry point (plan region, then partial-result region).
struct CallBuffers {
  kvx_pool* pool;
  const kvx::FixedScratch* fixed;
  uint8_t* base = nullptr;  // fixed scratch on the pool's device (after bind())

  // Bound on split parts of `per_part` bytes each.
  int64_t max_parts(size_t per_part) const {
    if (!fixed) return kMaxParts;
    return std::min<int64_t>(kMaxParts, (int64_t)(fixed->parts_bytes / per_part));
  }
  // Host-only size check of the plan (before any device call).
  int check_plan(size_t bytes) const {
    if (fixed && bytes > fixed->plan_bytes)
      return fail(KVX_EUNSUPPORTED, "work plan of %zu bytes exceeds the fixed scratch's %zu-byte plan region",
                  bytes, fixed->plan_bytes);
    return KVX_OK;
  }
  // With the pool's device current: the fixed scratch's address on it.
  int bind() {
    if (!fixed) return KVX_OK;
    void* p = nullptr;
    if (int rc = fixed->address(pool->device, &p)) return rc;
    base = (uint8_t*)p;
    return KVX_OK;
  }
  int parts(size_t bytes, hipStream_t s, float** out) {
    if (fixed) {
      if (bytes > fixed->parts_bytes)
        return fail(KVX_EUNSUPPORTED, "partial results of %zu bytes exceed the fixed scratch's %zu bytes", bytes,
                    fixed->parts_bytes);
      *out = (float*)(base + fixed->plan_bytes);
      return KVX_OK;
    }
    if (int rc = pool->parts.ensure(bytes, s)) return rc;
    *out = (float*)pool->parts.ptr;
    return KVX_OK;
  }
  int upload(const std::vector<uint8_t>& blob, hipStream_t s, void** out) {
    if (fixed) {
      // pageable source: the copy is staged before the call returns
      KVX_HIP(hipMemcpyAsync(base, blob.data(), blob.size(), hipMemcpyHostToDevice, s));
      *out = base;
      return KVX_OK;
    }
    return pool->st_attn.upload(blob.data(), blob.size(), s, out);
  }
  int done(hipStream_t s) {
    if (fixed) return KVX_OK;
    if (int rc = pool->st_attn.done(s)) return rc;
    return pool->parts.done(s);
  }
};

template <typename U, typename M>
std::vector<uint8_t> plan_blob(const std::vector<U>& units, const std::vector<M>& merges) {
  const size_t ub = units.size() * sizeof(U), mb = merges.size() * sizeof(M);
  std::vector<uint8_t> blob(ub + mb);
  if (ub) std::memcpy(blob.data(), units.data(), ub);
  if (mb) std::memcpy(blob.data() + ub, merges.data(), mb);
  return blob;
}

// The requests of a store batch in the kernel arguments when there are few enough
// (returns false otherwise: the unit list is uploaded instead).  Workgroup order
// matches the unit lists below: request by request, logical page by page.
bool inline_store_reqs(const kvx_batch* b, const std::vector<int64_t>& qo, kvx::StoreReqs& rq) {
  rq.n = 0;
  int32_t wg = 0;
  for (int r = 0; r < b->num_reqs; r++) {
    const int64_t P = b->prefix_lens[r], E = b->extend_lens[r];
    if (E == 0) continue;
    if (rq.n == kvx::kStoreInlineReqs) {
      rq.n = 0;
      return false;
    }
    const int64_t pages = (P + E - 1) / kvx::kPageSize - P / kvx::kPageSize + 1;
    rq.first[rq.n] = wg;
    rq.qo[rq.n] = (int32_t)qo[(size_t)r];
    rq.prefix[rq.n] = (int32_t)P;
    rq.end[rq.n] = (int32_t)(P + E);
    rq.page_base[rq.n] = b->page_indptr[r];
    wg += (int32_t)pages;
    rq.n++;
  }
  rq.first[rq.n] = wg;
  return rq.n > 0;
}

int decode_attention(kvx_pool* pool, const kvx_batch* batch, const std::vector<int64_t>& qo, const void* q,
                     int32_t num_q_heads, float sm_scale, void* out, float* lse, hipStream_t s, CallBuffers& buf) {
  const int D = pool->head_dim;
  constexpr int R = kvx::kDecodeMaxGroup;
  DecodePlan plan;
  if (int rc = make_decode_plan(batch, qo, pool->num_kv_heads, pool->split_keys,
                                buf.max_parts((size_t)R * (D + 1) * sizeof(float)), plan))
    return rc;
  const std::vector<uint8_t> blob = plan_blob(plan.units, plan.merges);
  if (int rc = buf.check_plan(blob.size())) return rc;
  if (int rc = use_device(pool)) return rc;
  if (validate_mode())
    if (int rc = check_page_ids(pool, batch, s)) return rc;
  if (int rc = buf.bind()) return rc;
  float* parts = nullptr;
  if (plan.n_parts > 0)
    if (int rc = buf.parts((size_t)plan.n_parts * R * (D + 1) * sizeof(float), s, &parts)) return rc;
  void* dev = nullptr;
  if (int rc = buf.upload(blob, s, &dev)) return rc;
  kvx::DecodeParams p;
  p.q = (const uint16_t*)q;
  p.out = (uint16_t*)out;
  p.lse = lse;
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.page_ids = batch->page_ids;
  p.units = (const DecodeUnit*)dev;
  p.o_part = plan.n_parts ? parts : nullptr;
  p.lse_part = plan.n_parts ? parts + (size_t)plan.n_parts * R * D : nullptr;
  p.k_scale = pool->scales_d;
  p.v_scale = pool->scales_d ? pool->scales_d + pool->num_kv_heads : nullptr;
  p.num_q_heads = num_q_heads;
  p.num_kv_heads = pool->num_kv_heads;
  p.group = num_q_heads / pool->num_kv_heads;
  p.scale_log2 = sm_scale * 1.4426950408889634f;
  hipError_t e = kvx::launch_decode(p, (int64_t)plan.units.size(), D, pool->kv_dtype == KVX_KV_FP8_E4M3, s);
  if (e != hipSuccess) return hip_fail(e, "decode kernel launch");
  if (!plan.merges.empty()) {
    kvx::DecodeMergeParams m;
    m.merges = (const DecodeMerge*)((const uint8_t*)dev + plan.units.size() * sizeof(DecodeUnit));
    m.o_part = p.o_part;
    m.lse_part = p.lse_part;
    m.out = (uint16_t*)out;
    m.lse = lse;
    m.num_q_heads = num_q_heads;
    m.group = p.group;
    e = kvx::launch_decode_merge(m, (int64_t)plan.merges.size(), D, s);
    if (e != hipSuccess) return hip_fail(e, "decode merge kernel launch");
  }
  return buf.done(s);
}

}  // namespace

extern "C" {

const char* kvx_last_error(void) { return g_last_error.c_str(); }

int kv_pool_set_split_keys(kvx_pool* pool, int32_t keys) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  if (keys < 0 || keys % kvx::kTileKeys != 0)
    return fail(KVX_EINVAL, "split keys %d: must be 0 or a positive multiple of %d", keys, kvx::kTileKeys);
  pool->split_keys = keys;
  return KVX_OK;
}

int kv_pool_set_scaled_q(kvx_pool* pool, int32_t enable) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  if (enable != 0 && enable != 1) return fail(KVX_EINVAL, "scaled_q %d: must be 0 or 1", enable);
  pool->scaled_q = enable;
  return KVX_OK;
}

int kv_pool_create(int64_t num_pages, int32_t page_size, int32_t num_kv_heads, int32_t head_dim,
                   int32_t kv_dtype, const float* k_scale, const float* v_scale, kvx_pool** out) {
  g_last_error.clear();
  if (out == nullptr) return fail(KVX_EINVAL, "out is NULL");
  *out = nullptr;
  if (num_pages <= 0) return fail(KVX_EINVAL, "num_pages = %lld must be > 0", (long long)num_pages);
  if (num_pages > (int64_t)INT32_MAX) return fail(KVX_EINVAL, "num_pages above 2^31-1");
  if (num_kv_heads <= 0) return fail(KVX_EINVAL, "num_kv_heads = %d must be > 0", num_kv_heads);
  if (num_kv_heads >= (1 << 15)) return fail(KVX_EUNSUPPORTED, "num_kv_heads too large");
  if (page_size != kvx::kPageSize) return fail(KVX_EUNSUPPORTED, "page_size %d (supported: 16)", page_size);
  if (head_dim != 64 && head_dim != 128) return fail(KVX_EUNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (kv_dtype != KVX_KV_BF16 && kv_dtype != KVX_KV_FP8_E4M3) return fail(KVX_EINVAL, "kv_dtype %d", kv_dtype);
  if (kv_dtype == KVX_KV_FP8_E4M3) {
    if (!k_scale || !v_scale) return fail(KVX_EUNSUPPORTED, "an fp8 pool needs k_scale and v_scale");
    for (int h = 0; h < num_kv_heads; h++)
      if (!(std::isfinite(k_scale[h]) && k_scale[h] > 0.f && std::isfinite(v_scale[h]) && v_scale[h] > 0.f))
        return fail(KVX_EINVAL, "fp8 scales of head %d must be finite and > 0", h);
  }
  const int eb = kv_dtype == KVX_KV_BF16 ? 2 : 1;
  const size_t bytes = (size_t)num_pages * num_kv_heads * page_size * head_dim * eb;
  if (bytes / (size_t)num_pages / (size_t)eb != (size_t)num_kv_heads * page_size * head_dim)
    return fail(KVX_EINVAL, "pool size overflows");
  kvx_pool* p = new kvx_pool();
  p->num_pages = num_pages;
  p->page_size = page_size;
  p->num_kv_heads = num_kv_heads;
  p->head_dim = head_dim;
  p->kv_dtype = kv_dtype;
  p->elem_bytes = eb;
  auto cleanup = [&](int rc) {
    if (p->k) (void)hipFree(p->k);
    if (p->v) (void)hipFree(p->v);
    if (p->scales_d) (void)hipFree(p->scales_d);
    delete p;
    return rc;
  };
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) return cleanup(hip_fail(e, "hipGetDevice"));
  e = hipMalloc(&p->k, bytes);
  if (e != hipSuccess) return cleanup(hip_fail(e, "hipMalloc(K pool)"));
  e = hipMalloc(&p->v, bytes);
  if (e != hipSuccess) return cleanup(hip_fail(e, "hipMalloc(V pool)"));
  e = hipMemset(p->k, 0, bytes);
  if (e == hipSuccess) e = hipMemset(p->v, 0, bytes);
  if (e != hipSuccess) return cleanup(hip_fail(e, "hipMemset(pool)"));
  if (kv_dtype == KVX_KV_FP8_E4M3) {
    std::vector<float> s((size_t)4 * num_kv_heads);
    for (int h = 0; h < num_kv_heads; h++) {
      s[(size_t)h] = k_scale[h];
      s[(size_t)num_kv_heads + h] = v_scale[h];
      s[(size_t)2 * num_kv_heads + h] = 1.0f / k_scale[h];  // fp32 reciprocal used to quantise
      s[(size_t)3 * num_kv_heads + h] = 1.0f / v_scale[h];
    }
    e = hipMalloc(&p->scales_d, s.size() * sizeof(float));
    if (e == hipSuccess) e = hipMemcpy(p->scales_d, s.data(), s.size() * sizeof(float), hipMemcpyHostToDevice);
    if (e != hipSuccess) return cleanup(hip_fail(e, "fp8 scales"));
  }
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return cleanup(hip_fail(e, "hipDeviceSynchronize"));
  *out = p;
  return KVX_OK;
}

int kv_pool_destroy(kvx_pool* pool) {
  g_last_error.clear();
  if (pool == nullptr) return KVX_OK;
  (void)use_device(pool);
  hipError_t e = hipDeviceSynchronize();
  pool->st_store.release();
  pool->st_attn.release();
  pool->st_io.release();
  pool->st_move.release();
  pool->parts.release();
  if (pool->k) (void)hipFree(pool->k);
  if (pool->v) (void)hipFree(pool->v);
  if (pool->scales_d) (void)hipFree(pool->scales_d);
  delete pool;
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  return KVX_OK;
}

int kv_pool_layout(const kvx_pool* pool, kvx_pool_layout* out) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  if (out == nullptr) return fail(KVX_EINVAL, "out is NULL");
  const int64_t S = pool->page_size, D = pool->head_dim, H = pool->num_kv_heads;
  std::memset(out, 0, sizeof *out);
  out->k_base = pool->k;
  out->v_base = pool->v;
  out->num_pages = pool->num_pages;
  out->page_size = pool->page_size;
  out->num_kv_heads = pool->num_kv_heads;
  out->head_dim = pool->head_dim;
  out->kv_dtype = pool->kv_dtype;
  out->elem_bytes = pool->elem_bytes;
  out->k_stride_page = H * S * D;
  out->k_stride_head = S * D;
  out->k_stride_slot = D;
  out->k_stride_dim = 1;
  out->v_stride_page = H * S * D;
  out->v_stride_head = S * D;
  out->v_stride_slot = 1;
  out->v_stride_dim = S;
  out->k_scale = pool->scales_d;
  out->v_scale = pool->scales_d ? pool->scales_d + H : nullptr;
  return KVX_OK;
}

static int page_io(kvx_pool* pool, const int32_t* page_ids, int64_t n, void* k_lin, void* v_lin, int to_pool,
                   kvx_stream_t stream) {
  if (int rc = check_pool(pool)) return rc;
  if (n < 0) return fail(KVX_EINVAL, "n = %lld < 0", (long long)n);
  if (n == 0) return KVX_OK;
  if (!page_ids || !k_lin || !v_lin) return fail(KVX_EINVAL, "page_ids, K and V buffers must be non-NULL");
  if (int rc = check_align(k_lin, "K buffer")) return rc;
  if (int rc = check_align(v_lin, "V buffer")) return rc;
  if (n > (int64_t)INT32_MAX) return fail(KVX_EINVAL, "too many pages");
  for (int64_t i = 0; i < n; i++)
    if (page_ids[i] < 0 || page_ids[i] >= pool->num_pages)
      return fail(KVX_ERANGE, "page_ids[%lld] = %d outside [0, %lld)", (long long)i, page_ids[i],
                  (long long)pool->num_pages);
  if (int rc = use_device(pool)) return rc;
  hipStream_t s = (hipStream_t)stream;
  void* ids_d = nullptr;
  if (int rc = pool->st_io.upload(page_ids, (size_t)n * sizeof(int32_t), s, &ids_d)) return rc;
  kvx::PageIoParams p;
  p.page_ids = (const int32_t*)ids_d;
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.k_lin = k_lin;
  p.v_lin = v_lin;
  p.num_kv_heads = pool->num_kv_heads;
  p.to_pool = to_pool;
  hipError_t e = kvx::launch_page_io(p, n, pool->head_dim, pool->elem_bytes, s);
  if (e != hipSuccess) return hip_fail(e, "page io kernel launch");
  return pool->st_io.done(s);
}

int kv_pool_write_pages(kvx_pool* pool, const int32_t* page_ids, int64_t n, const void* k_src, const void* v_src,
                        kvx_stream_t stream) {
  g_last_error.clear();
  return page_io(pool, page_ids, n, const_cast<void*>(k_src), const_cast<void*>(v_src), 1, stream);
}

int kv_pool_read_pages(const kvx_pool* pool, const int32_t* page_ids, int64_t n, void* k_dst, void* v_dst,
                       kvx_stream_t stream) {
  g_last_error.clear();
  return page_io(const_cast<kvx_pool*>(pool), page_ids, n, k_dst, v_dst, 0, stream);
}

static int64_t record_bytes(const kvx_pool* pool) {
  return 2 * (int64_t)pool->num_kv_heads * kvx::kPageSize * pool->head_dim * pool->elem_bytes;
}

int kv_pool_record_bytes(const kvx_pool* pool, int64_t* bytes) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  if (bytes == nullptr) return fail(KVX_EINVAL, "bytes is NULL");
  *bytes = record_bytes(pool);
  return KVX_OK;
}

// Spill (to_host) or reload whole pages between the pool and pinned host records.
static int page_move(kvx_pool* pool, const int32_t* page_ids, const int32_t* slots, int64_t n, const void* host,
                     int64_t host_slots, int to_host, kvx_stream_t stream) {
  if (int rc = check_pool(pool)) return rc;
  if (n < 0 || host_slots < 0) return fail(KVX_EINVAL, "n = %lld and host_slots = %lld must be >= 0", (long long)n,
                                           (long long)host_slots);
  if (n == 0) return KVX_OK;
  if (!page_ids || !slots || !host) return fail(KVX_EINVAL, "page_ids, slots and host must be non-NULL");
  if (int rc = check_align(host, "host")) return rc;
  if (n > (int64_t)INT32_MAX) return fail(KVX_EINVAL, "too many pages");
  for (int64_t i = 0; i < n; i++) {
    if (page_ids[i] < 0 || page_ids[i] >= pool->num_pages)
      return fail(KVX_ERANGE, "page_ids[%lld] = %d outside [0, %lld)", (long long)i, page_ids[i],
                  (long long)pool->num_pages);
    if (slots[i] < 0 || slots[i] >= host_slots)
      return fail(KVX_ERANGE, "slots[%lld] = %d outside [0, %lld)", (long long)i, slots[i], (long long)host_slots);
  }
  // the written side must not repeat: slots of a spill, pages of a reload
  std::vector<int32_t> dst(to_host ? slots : page_ids, (to_host ? slots : page_ids) + n);
  std::sort(dst.begin(), dst.end());
  if (std::adjacent_find(dst.begin(), dst.end()) != dst.end())
    return fail(KVX_EINVAL, "%s repeats an entry", to_host ? "slots" : "page_ids");
  if (int rc = use_device(pool)) return rc;
  hipPointerAttribute_t attr{};
  if (hipPointerGetAttributes(&attr, host) != hipSuccess || attr.type != hipMemoryTypeHost ||
      attr.devicePointer == nullptr) {
    (void)hipGetLastError();
    return fail(KVX_EINVAL, "host must be pinned host memory (hipHostMalloc, or a pinned torch tensor)");
  }
  const int64_t off = (const uint8_t*)host - (const uint8_t*)attr.hostPointer;
  hipStream_t s = (hipStream_t)stream;
  std::vector<int32_t> idx((size_t)(2 * n));
  std::copy(page_ids, page_ids + n, idx.begin());
  std::copy(slots, slots + n, idx.begin() + n);
  void* idx_d = nullptr;
  if (int rc = pool->st_move.upload(idx.data(), idx.size() * sizeof(int32_t), s, &idx_d)) return rc;
  kvx::PageMoveParams p;
  p.page_ids = (const int32_t*)idx_d;
  p.slots = (const int32_t*)idx_d + n;
  p.k_pool = (uint8_t*)pool->k;
  p.v_pool = (uint8_t*)pool->v;
  p.host = (uint8_t*)attr.devicePointer + (attr.hostPointer ? off : 0);
  p.block_bytes = record_bytes(pool) / 2;
  p.to_host = to_host;
  hipError_t e = kvx::launch_page_move(p, n, s);
  if (e != hipSuccess) return hip_fail(e, "page move kernel launch");
  return pool->st_move.done(s);
}

int kv_pool_spill(const kvx_pool* pool, const int32_t* page_ids, const int32_t* slots, int64_t n, void* host,
                  int64_t host_slots, kvx_stream_t stream) {
  g_last_error.clear();
  return page_move(const_cast<kvx_pool*>(pool), page_ids, slots, n, host, host_slots, 1, stream);
}

int kv_pool_reload(kvx_pool* pool, const int32_t* page_ids, const int32_t* slots, int64_t n, const void* host,
                   int64_t host_slots, kvx_stream_t stream) {
  g_last_error.clear();
  return page_move(pool, page_ids, slots, n, host, host_slots, 0, stream);
}

int store_kv(kvx_pool* pool, const kvx_batch* batch, const void* k_ext, const void* v_ext, kvx_stream_t stream) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  std::vector<int64_t> qo;
  if (int rc = check_batch(batch, qo)) return rc;
  if (qo.back() == 0) return KVX_OK;
  if (!k_ext || !v_ext) return fail(KVX_EINVAL, "k_ext and v_ext must be non-NULL");
  if (int rc = check_align(k_ext, "k_ext")) return rc;
  if (int rc = check_align(v_ext, "v_ext")) return rc;
  if (int rc = use_device(pool)) return rc;
  hipStream_t s = (hipStream_t)stream;
  if (validate_mode())
    if (int rc = check_page_ids(pool, batch, s)) return rc;
  std::vector<StoreUnit> units;
  const int S = kvx::kPageSize;
  for (int r = 0; r < batch->num_reqs; r++) {
    const int64_t P = batch->prefix_lens[r], E = batch->extend_lens[r];
    if (E == 0) continue;
    const int64_t L = P + E;
    for (int64_t lp = P / S; lp <= (L - 1) / S; lp++) {
      StoreUnit u;
      u.row_slot0 = (int32_t)(qo[(size_t)r] + lp * S - P);
      u.page_pos = (int32_t)(batch->page_indptr[r] + lp);
      u.slot_begin = (int32_t)(std::max<int64_t>(P, lp * S) - lp * S);
      u.slot_end = (int32_t)(std::min<int64_t>(L, lp * S + S) - lp * S);
      units.push_back(u);
    }
  }
  kvx::StoreParams p;
  void* units_d = nullptr;
  if (!inline_store_reqs(batch, qo, p.reqs))
    if (int rc = pool->st_store.upload(units.data(), units.size() * sizeof(StoreUnit), s, &units_d)) return rc;
  p.k_ext = (const uint16_t*)k_ext;
  p.v_ext = (const uint16_t*)v_ext;
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.page_ids = batch->page_ids;
  p.units = (const StoreUnit*)units_d;
  p.k_inv_scale = pool->scales_d ? pool->scales_d + 2 * pool->num_kv_heads : nullptr;
  p.v_inv_scale = pool->scales_d ? pool->scales_d + 3 * pool->num_kv_heads : nullptr;
  p.num_kv_heads = pool->num_kv_heads;
  hipError_t e = kvx::launch_store_kv(p, (int64_t)units.size(), pool->head_dim, pool->kv_dtype == KVX_KV_FP8_E4M3, s);
  if (e != hipSuccess) return hip_fail(e, "store_kv kernel launch");
  return p.reqs.n > 0 ? KVX_OK : pool->st_store.done(s);
}

int store_kv_rope(kvx_pool* pool, const kvx_batch* batch, const kvx_rope* rope, const void* q, int32_t num_q_heads,
                  void* q_out, const void* k_ext, const void* v_ext, kvx_stream_t stream) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  std::vector<int64_t> qo;
  if (int rc = check_batch(batch, qo)) return rc;
  if (rope == nullptr) return fail(KVX_EINVAL, "rope is NULL");
  const int D = pool->head_dim;
  const int rd = rope->rotary_dim;
  if (rd < 16 || rd > D || rd % 16 != 0)
    return fail(KVX_EINVAL, "rotary_dim = %d must be a multiple of 16 in [16, head_dim = %d]", rd, D);
  if (rope->style != KVX_ROPE_HALF && rope->style != KVX_ROPE_INTERLEAVED)
    return fail(KVX_EINVAL, "style = %d", rope->style);
  if (!(rope->norm_eps >= 0.0f) || !std::isfinite(rope->norm_eps))
    return fail(KVX_EINVAL, "norm_eps must be finite and >= 0");
  kvx::RopeParams p{};
  for (int j = 0; j < rd / 2; j++) {
    double f;
    if (rope->inv_freq) {
      f = rope->inv_freq[j];
      if (!(f >= 0.0) || !std::isfinite(f)) return fail(KVX_EINVAL, "inv_freq[%d] must be finite and >= 0", j);
    } else {
      if (!(rope->theta > 0.0) || !std::isfinite(rope->theta))
        return fail(KVX_EINVAL, "theta must be finite and > 0");
      f = std::pow(rope->theta, -2.0 * j / rd);
    }
    p.rev_freq[j] = f / 6.283185307179586476925286766559;  // turns per position
  }
  if (num_q_heads < 0) return fail(KVX_EINVAL, "num_q_heads = %d < 0", num_q_heads);
  if (num_q_heads > 0 && (!q || !q_out)) return fail(KVX_EINVAL, "q and q_out must be non-NULL");
  if (num_q_heads > 0) {
    if (int rc = check_align(q, "q")) return rc;
    if (int rc = check_align(q_out, "q_out")) return rc;
  }
  if (int rc = check_align(rope->q_norm, "q_norm")) return rc;
  if (int rc = check_align(rope->k_norm, "k_norm")) return rc;
  if (qo.back() == 0) return KVX_OK;
  if (!k_ext || !v_ext) return fail(KVX_EINVAL, "k_ext and v_ext must be non-NULL");
  if (int rc = check_align(k_ext, "k_ext")) return rc;
  if (int rc = check_align(v_ext, "v_ext")) return rc;
  if (int rc = use_device(pool)) return rc;
  hipStream_t s = (hipStream_t)stream;
  if (validate_mode())
    if (int rc = check_page_ids(pool, batch, s)) return rc;
  std::vector<kvx::RopeUnit> units;
  const int S = kvx::kPageSize;
  for (int r = 0; r < batch->num_reqs; r++) {
    const int64_t P = batch->prefix_lens[r], E = batch->extend_lens[r];
    if (E == 0) continue;
    const int64_t L = P + E;
    for (int64_t lp = P / S; lp <= (L - 1) / S; lp++) {
      kvx::RopeUnit u;
      u.row_slot0 = (int32_t)(qo[(size_t)r] + lp * S - P);
      u.page_pos = (int32_t)(batch->page_indptr[r] + lp);
      u.slot_begin = (int32_t)(std::max<int64_t>(P, lp * S) - lp * S);
      u.slot_end = (int32_t)(std::min<int64_t>(L, lp * S + S) - lp * S);
      u.pos_slot0 = (int32_t)(lp * S);
      units.push_back(u);
    }
  }
  void* units_d = nullptr;
  if (!inline_store_reqs(batch, qo, p.reqs))
    if (int rc = pool->st_store.upload(units.data(), units.size() * sizeof(kvx::RopeUnit), s, &units_d)) return rc;
  p.q = (const uint16_t*)q;
  p.q_out = (uint16_t*)q_out;
  p.k_ext = (const uint16_t*)k_ext;
  p.v_ext = (const uint16_t*)v_ext;
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.page_ids = batch->page_ids;
  p.units = (const kvx::RopeUnit*)units_d;
  p.k_inv_scale = pool->scales_d ? pool->scales_d + 2 * pool->num_kv_heads : nullptr;
  p.v_inv_scale = pool->scales_d ? pool->scales_d + 3 * pool->num_kv_heads : nullptr;
  p.q_norm = (const uint16_t*)rope->q_norm;
  p.k_norm = (const uint16_t*)rope->k_norm;
  p.num_q_heads = num_q_heads;
  p.num_kv_heads = pool->num_kv_heads;
  p.rotary_dim = rd;
  p.norm_eps = rope->norm_eps;
  hipError_t e = kvx::launch_store_kv_rope(p, (int64_t)units.size(), D, pool->kv_dtype == KVX_KV_FP8_E4M3,
                                           rope->style == KVX_ROPE_INTERLEAVED, s);
  if (e != hipSuccess) return hip_fail(e, "store_kv_rope kernel launch");
  return p.reqs.n > 0 ? KVX_OK : pool->st_store.done(s);
}

int extend_attention_plan(const kvx_batch* batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                          int32_t split_keys, kvx_work_item* items, int64_t cap, int64_t* count) {
  g_last_error.clear();
  if (count == nullptr) return fail(KVX_EINVAL, "count is NULL");
  *count = 0;
  if (int rc = check_heads(num_q_heads, num_kv_heads, head_dim)) return rc;
  if (split_keys < 0 || split_keys % kvx::kTileKeys != 0)
    return fail(KVX_EINVAL, "split keys %d: must be 0 or a positive multiple of %d", split_keys, kvx::kTileKeys);
  std::vector<int64_t> qo;
  if (int rc = check_batch(batch, qo, false)) return rc;
  if (cap < 0) return fail(KVX_EINVAL, "cap < 0");
  std::vector<kvx_work_item> out_items;
  if (qo.back() > 0) {
    if (is_decode_batch(batch, num_q_heads, num_kv_heads)) {
      DecodePlan dp;
      if (int rc = make_decode_plan(batch, qo, num_kv_heads, split_keys, kMaxParts, dp)) return rc;
      out_items = std::move(dp.items);
    } else {
      Plan plan;
      if (int rc = make_plan(batch, qo, num_q_heads, num_kv_heads, split_keys, kMaxParts, plan)) return rc;
      out_items = std::move(plan.items);
    }
  }
  *count = (int64_t)out_items.size();
  if (items != nullptr) {
    const int64_t m = std::min<int64_t>(cap, *count);
    for (int64_t i = 0; i < m; i++) items[i] = out_items[(size_t)i];
  }
  return KVX_OK;
}

int extend_attention(kvx_pool* pool, const kvx_batch* batch, const void* q, int32_t num_q_heads, float sm_scale,
                     void* out, float* lse, kvx_stream_t stream) {
  return kvx::attention_call(pool, batch, q, num_q_heads, sm_scale, out, lse, stream, nullptr);
}

}  // extern "C"

int kvx::attention_call(kvx_pool* pool, const kvx_batch* batch, const void* q, int32_t num_q_heads, float sm_scale,
                        void* out, float* lse, kvx_stream_t stream, const FixedScratch* fixed) {
  g_last_error.clear();
  if (int rc = check_pool(pool)) return rc;
  if (int rc = check_heads(num_q_heads, pool->num_kv_heads, pool->head_dim)) return rc;
  if (!(std::isfinite(sm_scale) && sm_scale > 0.f)) return fail(KVX_EINVAL, "sm_scale must be finite and > 0");
  std::vector<int64_t> qo;
  if (int rc = check_batch(batch, qo)) return rc;
  if (qo.back() == 0) return KVX_OK;
  if (!q || !out) return fail(KVX_EINVAL, "q and out must be non-NULL");
  if (int rc = check_align(q, "q")) return rc;
  if (int rc = check_align(out, "out")) return rc;
  if (lse != nullptr && ((uintptr_t)lse & 3u) != 0) return fail(KVX_EINVAL, "lse is not 4-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  CallBuffers buf{pool, fixed};

  if (is_decode_batch(batch, num_q_heads, pool->num_kv_heads))
    return decode_attention(pool, batch, qo, q, num_q_heads, sm_scale, out, lse, s, buf);

  const int D = pool->head_dim;
  const size_t part_bytes = (size_t)kvx::kTileRows * (D + 1) * sizeof(float);
  Plan plan;
  if (int rc = make_plan(batch, qo, num_q_heads, pool->num_kv_heads, pool->split_keys, buf.max_parts(part_bytes),
                         plan))
    return rc;
  // one upload: units, then merges
  const std::vector<uint8_t> blob = plan_blob(plan.units, plan.merges);
  if (int rc = buf.check_plan(blob.size())) return rc;
  if (int rc = use_device(pool)) return rc;
  if (validate_mode())
    if (int rc = check_page_ids(pool, batch, s)) return rc;
  if (int rc = buf.bind()) return rc;
  float* parts = nullptr;
  if (plan.n_parts > 0)
    if (int rc = buf.parts((size_t)plan.n_parts * part_bytes, s, &parts)) return rc;
  void* dev = nullptr;
  if (int rc = buf.upload(blob, s, &dev)) return rc;

  kvx::AttnParams p;
  p.q = (const uint16_t*)q;
  p.out = (uint16_t*)out;
  p.lse = lse;
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.page_ids = batch->page_ids;
  p.units = (const AttnUnit*)dev;
  p.o_part = plan.n_parts ? parts : nullptr;
  p.lse_part = plan.n_parts ? parts + (size_t)plan.n_parts * kvx::kTileRows * D : nullptr;
  p.k_scale = pool->scales_d;
  p.v_scale = pool->scales_d ? pool->scales_d + pool->num_kv_heads : nullptr;
  p.num_q_heads = num_q_heads;
  p.num_kv_heads = pool->num_kv_heads;
  p.group = num_q_heads / pool->num_kv_heads;
  p.tile_tok = kvx::kTileRows / p.group;
  p.scale_log2 = sm_scale * 1.4426950408889634f;
  hipError_t e = kvx::launch_extend_attention(p, (int64_t)plan.units.size(), D, pool->kv_dtype == KVX_KV_FP8_E4M3,
                                              pool->scaled_q != 0, s);
  if (e != hipSuccess) return hip_fail(e, "extend_attention kernel launch");
  if (!plan.merges.empty()) {
    kvx::MergeParams m;
    m.merges = (const MergeUnit*)((const uint8_t*)dev + plan.units.size() * sizeof(AttnUnit));
    m.o_part = p.o_part;
    m.lse_part = p.lse_part;
    m.out = (uint16_t*)out;
    m.lse = lse;
    m.num_q_heads = num_q_heads;
    m.group = p.group;
    e = kvx::launch_merge(m, (int64_t)plan.merges.size(), D, s);
    if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
  }
  return buf.done(s);
}
