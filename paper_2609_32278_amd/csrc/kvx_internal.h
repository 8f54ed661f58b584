// Internal declarations shared by the host code and the HIP kernels of libkvx.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kvx.h"

namespace kvx {

constexpr int kPageSize = 16;
constexpr int kTileRows = KVX_TILE_ROWS;  // query rows (token x query head of one KV head) per workgroup
constexpr int kTileKeys = 64;   // keys per K/V tile staged in LDS
constexpr int kAttnThreads = 512;  // 8 waves x 32 query rows
constexpr int kNumXcd = 8;      // L2 domains of an MI355X; workgroup i runs on XCD i % 8

// One attention workgroup: a tile of suffix tokens of one request and one KV head,
// over keys [key_begin, key_end) of the request's logical sequence.
struct AttnUnit {
  int32_t qo_row0;    // global suffix row of the tile's first token
  int32_t q_pos0;     // absolute position of that token (P + tok_begin)
  int32_t page_base;  // offset of the request's page list in page_ids
  int32_t key_begin;  // multiple of kTileKeys
  int32_t key_end;    // exclusive; key_end <= key_begin marks a padding entry
  int32_t head_ntok;  // (kv_head << 16) | tokens in the tile
  int32_t part;       // -1: final result; else index of this part's partial result
  int32_t req;
};
static_assert(sizeof(AttnUnit) == 32, "AttnUnit is 32 bytes");

// Log-sum-exp merge of the parts of one split tile.
struct MergeUnit {
  int32_t qo_row0;
  int32_t head_ntok;
  int32_t part0;
  int32_t nparts;
};

// One KV-store workgroup: the suffix slots [slot_begin, slot_end) of one page.
struct StoreUnit {
  int32_t row_slot0;  // suffix row that slot 0 of the page would hold (may be negative)
  int32_t page_pos;   // index into page_ids
  int32_t slot_begin;
  int32_t slot_end;
};

struct AttnParams {
  const uint16_t* q;      // bf16 [T, Hq, D]
  uint16_t* out;          // bf16 [T, Hq, D]
  float* lse;             // fp32 [T, Hq] or null
  const void* k_pool;
  const void* v_pool;
  const int32_t* page_ids;
  const AttnUnit* units;
  float* o_part;          // fp32 [parts, kTileRows, D]
  float* lse_part;        // fp32 [parts, kTileRows]
  const float* k_scale;   // fp8 pool: device [Hkv]
  const float* v_scale;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;          // Hq / Hkv
  int32_t tile_tok;       // tokens per tile = kTileRows / group
  float scale_log2;       // sm_scale * log2(e)
};

struct MergeParams {
  const MergeUnit* merges;
  const float* o_part;
  const float* lse_part;
  uint16_t* out;
  float* lse;
  int32_t num_q_heads;
  int32_t group;
};

// The requests of a small store batch, passed by value in the kernel arguments so
// that no unit list is uploaded: request r's pages are the workgroups
// [first[r], first[r + 1]), logical pages prefix[r] / 16 onwards.
constexpr int kStoreInlineReqs = 96;
struct StoreReqs {
  int32_t n;                            // requests with work; 0: use the uploaded unit list
  int32_t first[kStoreInlineReqs + 1];  // first workgroup of each request; first[n] = all
  int32_t qo[kStoreInlineReqs];         // suffix row of the request's first suffix token
  int32_t prefix[kStoreInlineReqs];     // P
  int32_t end[kStoreInlineReqs];        // P + E
  int32_t page_base[kStoreInlineReqs];  // page_indptr[r]
};

struct StoreParams {
  const uint16_t* k_ext;  // bf16 [T, Hkv, D]
  const uint16_t* v_ext;
  void* k_pool;
  void* v_pool;
  const int32_t* page_ids;
  const StoreUnit* units;
  const float* k_inv_scale;  // fp8 pool: device [Hkv], fp32 1/scale
  const float* v_inv_scale;
  int32_t num_kv_heads;
  StoreReqs reqs;            // reqs.n > 0: the units come from here instead
};

// One fused-store workgroup: a StoreUnit plus the absolute position of slot 0.
struct RopeUnit {
  int32_t row_slot0;
  int32_t page_pos;
  int32_t slot_begin;
  int32_t slot_end;
  int32_t pos_slot0;  // position t of slot 0 of the page (a multiple of 16)
};

constexpr int kRopeMaxPlanes = 64;  // rotary_dim / 2 <= head_dim / 2

struct RopeParams {
  const uint16_t* q;      // bf16 [T, Hq, D], or null when num_q_heads == 0
  uint16_t* q_out;        // may equal q
  const uint16_t* k_ext;  // bf16 [T, Hkv, D]
  const uint16_t* v_ext;
  void* k_pool;
  void* v_pool;
  const int32_t* page_ids;
  const RopeUnit* units;
  const float* k_inv_scale;  // fp8 pool: device [Hkv], fp32 1/scale
  const float* v_inv_scale;
  const uint16_t* q_norm;    // bf16 [D] RMS-norm weights, or null
  const uint16_t* k_norm;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t rotary_dim;        // multiple of 16, <= D
  float norm_eps;
  double rev_freq[kRopeMaxPlanes];  // plane rate in revolutions per position: f_j / (2 pi)
  StoreReqs reqs;                   // reqs.n > 0: the units come from here instead
};

struct PageIoParams {
  const int32_t* page_ids;  // device [n]
  void* k_pool;
  void* v_pool;
  void* k_lin;              // canonical [n][Hkv][16][D] buffers
  void* v_lin;
  int32_t num_kv_heads;
  int32_t to_pool;          // 1: write pages into the pool, 0: read them out
};

// Raw page records between the pool and host memory: record i = the K block then
// the V block of page page_ids[i], at host + slots[i] * 2 * block_bytes.
struct PageMoveParams {
  const int32_t* page_ids;  // device [n]
  const int32_t* slots;     // device [n]
  uint8_t* k_pool;
  uint8_t* v_pool;
  uint8_t* host;            // device-accessible address of pinned host memory
  int64_t block_bytes;      // Hkv * 16 * D * elem bytes (a multiple of 1 KiB)
  int32_t to_host;          // 1: pool -> host (spill), 0: host -> pool (reload)
};

// ---- decode (one query token per request): a key chunk of one (request, KV head)
constexpr int kDecodeThreads = 256;  // 4 waves, each streaming every 4th pair of pages
constexpr int kDecodeMaxGroup = 16;  // query heads per KV head held in one MFMA column block
constexpr int kDecodeChunkAlign = 64;  // chunk boundaries are multiples of it (keys)

struct DecodeUnit {
  int32_t qo_row;     // the request's only suffix row
  int32_t page_base;  // offset of the request's page list in page_ids
  int32_t key_begin;  // multiple of kDecodeChunkAlign
  int32_t key_end;    // exclusive
  int32_t head;       // KV head
  int32_t part;       // -1: final result; else index of this chunk's partial result
  int32_t req;
  int32_t pad;
};
static_assert(sizeof(DecodeUnit) == 32, "DecodeUnit is 32 bytes");

struct DecodeMerge {
  int32_t qo_row;
  int32_t head;
  int32_t part0;
  int32_t nparts;
};

struct DecodeParams {
  const uint16_t* q;      // bf16 [T, Hq, D]
  uint16_t* out;          // bf16 [T, Hq, D]
  float* lse;             // fp32 [T, Hq] or null
  const void* k_pool;     // [page][kv_head][slot][D], bf16 or fp8
  const void* v_pool;     // [page][kv_head][D][slot]
  const int32_t* page_ids;
  const DecodeUnit* units;
  float* o_part;          // fp32 [parts, kDecodeMaxGroup, D]
  float* lse_part;        // fp32 [parts, kDecodeMaxGroup]
  const float* k_scale;   // fp8 pool: device [Hkv]
  const float* v_scale;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;          // Hq / Hkv <= kDecodeMaxGroup
  float scale_log2;
};

struct DecodeMergeParams {
  const DecodeMerge* merges;
  const float* o_part;
  const float* lse_part;
  uint16_t* out;
  float* lse;
  int32_t num_q_heads;
  int32_t group;
};

hipError_t launch_decode(const DecodeParams& p, int64_t n_units, int head_dim, bool fp8, hipStream_t stream);
hipError_t launch_decode_merge(const DecodeMergeParams& p, int64_t n_merges, int head_dim, hipStream_t stream);

// Record a failure for kvx_last_error() and return `code` (host code of any file).
int report(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Fixed device scratch of the allocation-free attention entry point: a plan region
// of plan_bytes followed by a partial-result region of parts_bytes, at an address
// that `address` gives per device (called with that device current).
struct FixedScratch {
  size_t plan_bytes;
  size_t parts_bytes;
  int (*address)(int device, void** base);
};

// extend_attention's whole call: argument checks, plan, upload, launches.  With
// fixed == nullptr the plan goes through the pool's staging buffer and split
// parts into its growable workspace; otherwise both go into the fixed scratch,
// the plan is bounded by its regions (EUNSUPPORTED beyond them, checked on the
// host before any device call) and nothing is allocated.
int attention_call(kvx_pool* pool, const kvx_batch* batch, const void* q, int32_t num_q_heads, float sm_scale,
                   void* out, float* lse, kvx_stream_t stream, const FixedScratch* fixed);

hipError_t launch_extend_attention(const AttnParams& p, int64_t n_units, int head_dim, bool fp8, bool scaled_q,
                                   hipStream_t stream);
hipError_t launch_merge(const MergeParams& p, int64_t n_merges, int head_dim, hipStream_t stream);
hipError_t launch_store_kv(const StoreParams& p, int64_t n_units, int head_dim, bool fp8,
                           hipStream_t stream);
hipError_t launch_store_kv_rope(const RopeParams& p, int64_t n_units, int head_dim, bool fp8, bool interleaved,
                                hipStream_t stream);
hipError_t launch_page_move(const PageMoveParams& p, int64_t n_pages, hipStream_t stream);
hipError_t launch_page_io(const PageIoParams& p, int64_t n_pages, int head_dim, int elem_bytes,
                          hipStream_t stream);

}  // namespace kvx
