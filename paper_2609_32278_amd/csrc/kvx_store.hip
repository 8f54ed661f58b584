// KV store into the paged pool and raw page I/O, gfx950 (CDNA4).
//
// Prefill materialises the suffix's K/V in every attention layer (paper,
// Section 2); store_kv writes them into the request's pages so that the next
// attention pass -- and every later turn that reuses this prefix -- reads them
// from the pool.  HBM-bound: each element is read once and written once.
//
// Pool layout: K [page][kv_head][slot][dim], V [page][kv_head][dim][slot].
// One workgroup handles one page of one request for one group of 4 KV heads
// (head_dim 128) or 8 (head_dim 64) -- grid x = the page, y = the head group, so
// that a batch touching few pages still fills the chip -- and issues all of its
// loads before using any (four K and four V 16-byte loads in flight per thread):
// K rows are copied with 16-byte accesses, V rows are staged in LDS and written
// out transposed, one 16-slot column (32 bytes bf16 / 16 bytes fp8) per dim.
// fp8 pool: code = e4m3_rne(clamp(x * inv_scale_h, -448, 448)) with the
// hardware converter v_cvt_pk_fp8_f32 (OCP e4m3 on gfx950).

#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int kStoreThreads = 256;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ float clamp448(float x) { return fminf(fmaxf(x, -448.0f), 448.0f); }

// 4 floats -> 4 e4m3 codes (byte i = value i)
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  int r = __builtin_amdgcn_cvt_pk_fp8_f32(clamp448(a), clamp448(b), 0, false);
  r = __builtin_amdgcn_cvt_pk_fp8_f32(clamp448(c), clamp448(d), r, true);
  return (uint32_t)r;
}

// Write the staged V rows vs[slot][dim] of one (page, head) block as the pool's
// [dim][slot] columns, 8 slots per thread and step (16 bytes bf16 / 8 bytes fp8);
// only slots in [slot_begin, slot_end) are written.
template <int D, bool FP8>
__device__ __forceinline__ void write_vt(const uint16_t (&vs)[kPageSize][D + 8], void* v_pool, size_t blk,
                                         int slot_begin, int slot_end, float vinv) {
  const bool full = slot_begin == 0 && slot_end == kPageSize;
  for (int c = threadIdx.x; c < 2 * D; c += kStoreThreads) {
    const int d = c / 2, half = c % 2;
    const int s0 = half * 8;
    if (s0 + 8 <= slot_begin || s0 >= slot_end) continue;
    float x[8];
    uint16_t raw[8];
#pragma unroll
    for (int e = 0; e < 8; e++) {
      raw[e] = vs[s0 + e][d];
      x[e] = bf16_to_f32(raw[e]) * vinv;
    }
    const bool whole = full || (s0 >= slot_begin && s0 + 8 <= slot_end);
    if constexpr (FP8) {
      uint8_t* dst = (uint8_t*)v_pool + blk + (size_t)d * kPageSize + s0;
      uint2 code;
      code.x = e4m3x4(x[0], x[1], x[2], x[3]);
      code.y = e4m3x4(x[4], x[5], x[6], x[7]);
      if (whole) {
        *(uint2*)dst = code;
      } else {
        const uint8_t* cb = (const uint8_t*)&code;
        for (int e = 0; e < 8; e++)
          if (s0 + e >= slot_begin && s0 + e < slot_end) dst[e] = cb[e];
      }
    } else {
      uint16_t* dst = (uint16_t*)v_pool + blk + (size_t)d * kPageSize + s0;
      if (whole) {
        uint4 w;
        w.x = raw[0] | ((uint32_t)raw[1] << 16);
        w.y = raw[2] | ((uint32_t)raw[3] << 16);
        w.z = raw[4] | ((uint32_t)raw[5] << 16);
        w.w = raw[6] | ((uint32_t)raw[7] << 16);
        *(uint4*)dst = w;
      } else {
        for (int e = 0; e < 8; e++)
          if (s0 + e >= slot_begin && s0 + e < slot_end) dst[e] = raw[e];
      }
    }
  }
}

// The unit of workgroup b of a small batch (see StoreReqs); uniform.
__device__ __forceinline__ RopeUnit inline_unit(const StoreReqs& rq, int b) {
  int lo = 0, hi = rq.n;  // request r with first[r] <= b < first[r + 1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (rq.first[mid] <= b) lo = mid;
    else hi = mid;
  }
  const int P = rq.prefix[lo], L = rq.end[lo];
  const int lp = P / kPageSize + (b - rq.first[lo]);
  RopeUnit u;
  u.pos_slot0 = lp * kPageSize;
  u.row_slot0 = rq.qo[lo] + u.pos_slot0 - P;
  u.page_pos = rq.page_base[lo] + lp;
  u.slot_begin = (P > u.pos_slot0 ? P : u.pos_slot0) - u.pos_slot0;
  u.slot_end = (L < u.pos_slot0 + kPageSize ? L : u.pos_slot0 + kPageSize) - u.pos_slot0;
  return u;
}

template <int D, bool FP8>
__global__ __launch_bounds__(kStoreThreads) void store_kv_kernel(StoreParams p) {
  constexpr int CPR = D / 8;                          // 16-byte chunks per bf16 row
  constexpr int CHUNKS = kPageSize * CPR;             // per head
  constexpr int HB = 4 * kStoreThreads / CHUNKS;      // heads per pass: 4 (D = 128), 8 (D = 64)
  constexpr int PER = HB * CHUNKS / kStoreThreads;    // chunks per thread and pass
  static_assert(PER == 4, "four K and four V loads in flight per thread");
  // V rows of this page for the pass's heads, staged for the transpose: [head][16 slots][D] bf16
  __shared__ __attribute__((aligned(16))) uint16_t vs[HB][kPageSize][D + 8];
  StoreUnit su;
  if (p.reqs.n > 0) {
    const RopeUnit u = inline_unit(p.reqs, blockIdx.x);
    su = StoreUnit{u.row_slot0, u.page_pos, u.slot_begin, u.slot_end};
  } else {
    su = p.units[blockIdx.x];
  }
  const int page = p.page_ids[su.page_pos];
  const int H = p.num_kv_heads;

  {
    const int h0 = blockIdx.y * HB;
    // every load of the pass is issued before any of them is used
    uint4 kx[PER], vx[PER];
#pragma unroll
    for (int j = 0; j < PER; j++) {
      const int i = threadIdx.x + j * kStoreThreads;
      const int hd = h0 + i / CHUNKS, slot = (i % CHUNKS) / CPR, cc = i % CPR;
      kx[j] = vx[j] = make_uint4(0, 0, 0, 0);
      if (hd < H && slot >= su.slot_begin && slot < su.slot_end) {
        const size_t src = ((size_t)(su.row_slot0 + slot) * H + hd) * D + cc * 8;
        kx[j] = *(const uint4*)(p.k_ext + src);
        vx[j] = *(const uint4*)(p.v_ext + src);
      }
    }
#pragma unroll
    for (int j = 0; j < PER; j++) {
      const int i = threadIdx.x + j * kStoreThreads;
      const int hb = i / CHUNKS, hd = h0 + hb, slot = (i % CHUNKS) / CPR, cc = i % CPR;
      if (hd >= H) continue;
      if (slot >= su.slot_begin && slot < su.slot_end) {
        const size_t blk = ((size_t)page * H + hd) * (size_t)(kPageSize * D);
        if constexpr (FP8) {
          const float kinv = p.k_inv_scale[hd];
          const uint16_t* ke = (const uint16_t*)&kx[j];
          uint2 code;
          code.x = e4m3x4(bf16_to_f32(ke[0]) * kinv, bf16_to_f32(ke[1]) * kinv,
                          bf16_to_f32(ke[2]) * kinv, bf16_to_f32(ke[3]) * kinv);
          code.y = e4m3x4(bf16_to_f32(ke[4]) * kinv, bf16_to_f32(ke[5]) * kinv,
                          bf16_to_f32(ke[6]) * kinv, bf16_to_f32(ke[7]) * kinv);
          *(uint2*)((uint8_t*)p.k_pool + blk + (size_t)slot * D + cc * 8) = code;
        } else {
          *(uint4*)((uint16_t*)p.k_pool + blk + (size_t)slot * D + cc * 8) = kx[j];
        }
      }
      *(uint4*)(&vs[hb][slot][cc * 8]) = vx[j];
    }
    __syncthreads();
    for (int hb = 0; hb < HB && h0 + hb < H; hb++) {
      const int hd = h0 + hb;
      const size_t blk = ((size_t)page * H + hd) * (size_t)(kPageSize * D);
      write_vt<D, FP8>(vs[hb], p.v_pool, blk, su.slot_begin, su.slot_end, FP8 ? p.v_inv_scale[hd] : 1.0f);
    }
  }
}

// ---------------------------------------------------------------- fused RoPE store
//
// The step before attention, fused into the store (the models the paper serves
// normalise and rotate Q and K before K is cached; the paper itself describes
// neither step): every Q and K head row of the unit's tokens is optionally
// RMS-normalised, rotated by its absolute position, and then written -- Q to
// q_out as bf16, K into the pool as store_kv would store it.  V is stored as by
// store_kv.  Arithmetic is fp32; each angle is reduced to [-pi, pi] in fp64 from
// the plane's rate in revolutions per position, so positions far past 2^24
// keep full precision.  Results are rounded once (RNE bf16 or e4m3).
//
// A head row of D bf16 values is D/8 16-byte chunks held by D/8 consecutive
// lanes; the RMS sum is reduced across those lanes, and in the half layout a
// chunk of the first half meets its plane partners in the chunk rotary_dim/16
// lanes further on (one lane shuffle per value).

constexpr int kRopeBatch = 4;  // chunks per thread loaded before any is processed

template <int D, bool INTERLEAVED>
struct RopeLane {
  static constexpr int CPR = D / 8;
  int cc;           // chunk of the row this lane handles (fixed for the thread)
  int partner;      // lane holding the plane partners (half layout)
  int jb;           // first plane of the chunk
  bool rot;         // the chunk lies inside rotary_dim
  float sgn;        // half layout: -1 for the plane's first dims, +1 for its second

  __device__ RopeLane(int rotary_dim) {
    cc = threadIdx.x % CPR;
    const int lane = threadIdx.x & 63;
    if constexpr (INTERLEAVED) {
      rot = cc < (rotary_dim >> 3);
      jb = 4 * cc;
      partner = lane;
      sgn = 0.0f;
    } else {
      const int r16 = rotary_dim >> 4;
      const bool first = cc < r16;
      rot = cc < 2 * r16;
      jb = first ? 8 * cc : 8 * (cc - r16);
      partner = lane + (first ? r16 : (rot ? -r16 : 0));
      sgn = first ? -1.0f : 1.0f;
    }
  }
};

// x: the 8 values of this lane's chunk of one row at `slot`; in place -> rotated.
// Every lane of the row must execute this (shuffles).
template <int D, bool INTERLEAVED>
__device__ __forceinline__ void rope_chunk(float (&x)[8], const RopeLane<D, INTERLEAVED>& rl,
                                           const float2* cs_slot) {
  if constexpr (INTERLEAVED) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const float2 t = rl.rot ? cs_slot[rl.jb + i] : make_float2(1.0f, 0.0f);
      const float a = x[2 * i], b = x[2 * i + 1];
      x[2 * i] = a * t.x - b * t.y;
      x[2 * i + 1] = a * t.y + b * t.x;
    }
  } else {
    float pe[8];
#pragma unroll
    for (int e = 0; e < 8; e++) pe[e] = __shfl(x[e], rl.partner, 64);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      const float2 t = rl.rot ? cs_slot[rl.jb + e] : make_float2(1.0f, 0.0f);
      // first dims: a cos - b sin (b = partner); second dims: b cos + a sin (a = partner)
      x[e] = x[e] * t.x + rl.sgn * (pe[e] * t.y);
    }
  }
}

// Normalise and rotate the n_rows head rows at src ([row][D] bf16; row = tok *
// heads + head, token tok at slot slot_begin + tok) and hand each chunk's
// results to out(row, chunk, y).
template <int D, bool INTERLEAVED, class Out>
__device__ __forceinline__ void rope_rows(const uint16_t* __restrict__ src, int n_rows, int heads,
                                          int slot_begin, const float2 (*cs)[kRopeMaxPlanes],
                                          const uint16_t* norm_w, float eps, int rotary_dim, Out&& out) {
  constexpr int CPR = D / 8;
  const int n = n_rows * CPR;
  const RopeLane<D, INTERLEAVED> rl(rotary_dim);
  float w[8];
  if (norm_w) {
    const uint4 wr = *(const uint4*)(norm_w + rl.cc * 8);
    const uint16_t* wh = (const uint16_t*)&wr;
#pragma unroll
    for (int e = 0; e < 8; e++) w[e] = bf16_to_f32(wh[e]);
  }
  for (int c0 = threadIdx.x; c0 < n; c0 += kRopeBatch * kStoreThreads) {
    uint4 raw[kRopeBatch];
#pragma unroll
    for (int b = 0; b < kRopeBatch; b++) {
      const int c = c0 + b * kStoreThreads;
      raw[b] = c < n ? *(const uint4*)(src + (size_t)c * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int b = 0; b < kRopeBatch; b++) {
      const int c = c0 + b * kStoreThreads;
      const int row = c / CPR;
      const uint16_t* h16 = (const uint16_t*)&raw[b];
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; e++) x[e] = bf16_to_f32(h16[e]);
      if (norm_w) {
        float ss = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; e++) ss = fmaf(x[e], x[e], ss);
#pragma unroll
        for (int m = 1; m < CPR; m <<= 1) ss += __shfl_xor(ss, m, 64);
        const float inv = 1.0f / sqrtf(ss * (1.0f / D) + eps);
#pragma unroll
        for (int e = 0; e < 8; e++) x[e] = (x[e] * inv) * w[e];
      }
      const int slot = slot_begin + (c < n ? row / heads : 0);
      rope_chunk<D, INTERLEAVED>(x, rl, cs[slot]);
      if (c < n) out(row, rl.cc, x);
    }
  }
}

__device__ __forceinline__ uint4 pack_bf16x8(const float (&y)[8]) {
  uint4 r;
  uint32_t* w = (uint32_t*)&r;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const __bf16 lo = (__bf16)y[2 * i], hi = (__bf16)y[2 * i + 1];
    w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
  }
  return r;
}

template <int D, bool FP8, bool INTERLEAVED>
__global__ __launch_bounds__(kStoreThreads) void store_kv_rope_kernel(RopeParams p) {
  __shared__ float2 cs[kPageSize][kRopeMaxPlanes];  // (cos, sin) of every live slot and plane
  __shared__ __attribute__((aligned(16))) uint16_t vs[kPageSize][D + 8];
  const RopeUnit u = p.reqs.n > 0 ? inline_unit(p.reqs, blockIdx.x) : p.units[blockIdx.x];
  const int page = p.page_ids[u.page_pos];
  const int planes = p.rotary_dim / 2;
  const int ntok = u.slot_end - u.slot_begin;

  for (int e = threadIdx.x; e < ntok * planes; e += kStoreThreads) {
    const int s = u.slot_begin + e / planes, j = e % planes;
    double rev = (double)(u.pos_slot0 + s) * p.rev_freq[j];  // exact position times the rate
    rev -= rint(rev);                                          // [-1/2, 1/2] turn, exact
    float sn, cn;
    sincospif(2.0f * (float)rev, &sn, &cn);
    cs[s][j] = make_float2(cn, sn);
  }
  __syncthreads();

  constexpr int CPR = D / 8;
  const int Hq = p.num_q_heads, H = p.num_kv_heads;
  const int row0 = u.row_slot0 + u.slot_begin;  // first suffix row of the unit
  if (Hq > 0) {
    const size_t base = (size_t)row0 * Hq * D;
    uint16_t* qo = p.q_out + base;
    rope_rows<D, INTERLEAVED>(p.q + base, ntok * Hq, Hq, u.slot_begin, cs, p.q_norm, p.norm_eps, p.rotary_dim,
                              [&](int row, int cc, const float(&y)[8]) {
                                *(uint4*)(qo + (size_t)row * D + cc * 8) = pack_bf16x8(y);
                              });
  }
  rope_rows<D, INTERLEAVED>(
      p.k_ext + (size_t)row0 * H * D, ntok * H, H, u.slot_begin, cs, p.k_norm, p.norm_eps, p.rotary_dim,
      [&](int row, int cc, const float(&y)[8]) {
        const int hd = row % H, slot = u.slot_begin + row / H;
        const size_t blk = ((size_t)page * H + hd) * (size_t)(kPageSize * D);
        if constexpr (FP8) {
          const float kinv = p.k_inv_scale[hd];
          uint2 code;
          code.x = e4m3x4(y[0] * kinv, y[1] * kinv, y[2] * kinv, y[3] * kinv);
          code.y = e4m3x4(y[4] * kinv, y[5] * kinv, y[6] * kinv, y[7] * kinv);
          *(uint2*)((uint8_t*)p.k_pool + blk + (size_t)slot * D + cc * 8) = code;
        } else {
          *(uint4*)((uint16_t*)p.k_pool + blk + (size_t)slot * D + cc * 8) = pack_bf16x8(y);
        }
      });

  // V: staged per head in LDS and written as [dim][slot] columns
  for (int hd = 0; hd < H; hd++) {
    for (int c = threadIdx.x; c < kPageSize * CPR; c += kStoreThreads) {
      const int slot = c / CPR, cc = c % CPR;
      uint4 vx = make_uint4(0, 0, 0, 0);
      if (slot >= u.slot_begin && slot < u.slot_end)
        vx = *(const uint4*)(p.v_ext + ((size_t)(u.row_slot0 + slot) * H + hd) * D + cc * 8);
      *(uint4*)(&vs[slot][cc * 8]) = vx;
    }
    __syncthreads();
    const size_t blk = ((size_t)page * H + hd) * (size_t)(kPageSize * D);
    write_vt<D, FP8>(vs, p.v_pool, blk, u.slot_begin, u.slot_end, FP8 ? p.v_inv_scale[hd] : 1.0f);
    __syncthreads();
  }
}

// Spill / reload of whole pages between the pool and pinned host memory.  One
// workgroup per (page, K|V block): the block is contiguous on both sides, so
// every lane moves 16-byte pieces, four in flight before any store (host memory
// is reached over the host link: latency is long, concurrency hides it).
__global__ __launch_bounds__(256) void page_move_kernel(PageMoveParams p) {
  constexpr int kUnroll = 4;
  const int i = blockIdx.x;
  const int kv = blockIdx.y;  // 0: K block, 1: V block
  const int64_t page = p.page_ids[i];
  uint8_t* dev = (kv == 0 ? p.k_pool : p.v_pool) + page * p.block_bytes;
  uint8_t* host = p.host + ((int64_t)p.slots[i] * 2 + kv) * p.block_bytes;
  const uint8_t* src = p.to_host ? dev : host;
  uint8_t* dst = p.to_host ? host : dev;
  const int64_t pieces = p.block_bytes / 16;
  for (int64_t c0 = threadIdx.x; c0 < pieces; c0 += kUnroll * 256) {
    uint4 x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; u++) {
      const int64_t c = c0 + u * 256;
      if (c < pieces) x[u] = *(const uint4*)(src + c * 16);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; u++) {
      const int64_t c = c0 + u * 256;
      if (c < pieces) *(uint4*)(dst + c * 16) = x[u];
    }
  }
}

// Raw page copy between canonical [n][Hkv][16][D] buffers and the pool.
template <int D, int EB>
__global__ __launch_bounds__(256) void page_io_kernel(PageIoParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t tile[kPageSize][D * EB + 16];
  const int i = blockIdx.x;
  const int hd = blockIdx.y;
  const int page = p.page_ids[i];
  const size_t elems = (size_t)kPageSize * D;
  const size_t lin = ((size_t)i * p.num_kv_heads + hd) * elems * EB;
  const size_t pool = ((size_t)page * p.num_kv_heads + hd) * elems * EB;
  constexpr int ROWB = D * EB;  // bytes per [slot] row of K / canonical V
  constexpr int CH = ROWB / 16; // 16-byte chunks per row
  // K: same layout on both sides
  for (int c = threadIdx.x; c < kPageSize * CH; c += blockDim.x) {
    const size_t off = (size_t)c * 16;
    if (p.to_pool) *(uint4*)((uint8_t*)p.k_pool + pool + off) = *(const uint4*)((const uint8_t*)p.k_lin + lin + off);
    else *(uint4*)((uint8_t*)p.k_lin + lin + off) = *(const uint4*)((const uint8_t*)p.k_pool + pool + off);
  }
  // V: canonical [slot][dim] <-> pool [dim][slot], through LDS
  if (p.to_pool) {
    for (int c = threadIdx.x; c < kPageSize * CH; c += blockDim.x) {
      const int s = c / CH, cc = c % CH;
      *(uint4*)&tile[s][cc * 16] = *(const uint4*)((const uint8_t*)p.v_lin + lin + (size_t)s * ROWB + cc * 16);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < (int)elems; e += blockDim.x) {
      const int d = e / kPageSize, s = e % kPageSize;
      uint8_t* dst = (uint8_t*)p.v_pool + pool + (size_t)e * EB;
      for (int b = 0; b < EB; b++) dst[b] = tile[s][d * EB + b];
    }
  } else {
    for (int e = threadIdx.x; e < (int)elems; e += blockDim.x) {
      const int d = e / kPageSize, s = e % kPageSize;
      const uint8_t* src = (const uint8_t*)p.v_pool + pool + (size_t)e * EB;
      for (int b = 0; b < EB; b++) tile[s][d * EB + b] = src[b];
    }
    __syncthreads();
    for (int c = threadIdx.x; c < kPageSize * CH; c += blockDim.x) {
      const int s = c / CH, cc = c % CH;
      *(uint4*)((uint8_t*)p.v_lin + lin + (size_t)s * ROWB + cc * 16) = *(const uint4*)&tile[s][cc * 16];
    }
  }
}

}  // namespace

hipError_t launch_store_kv(const StoreParams& p, int64_t n_units, int head_dim, bool fp8,
                           hipStream_t stream) {
  if (n_units <= 0) return hipSuccess;
  const int hb = head_dim == 128 ? 4 : 8;  // heads per workgroup (HB of the kernel)
  dim3 grid((unsigned)n_units, (unsigned)((p.num_kv_heads + hb - 1) / hb)), block(kStoreThreads);
  if (head_dim == 128) {
    if (fp8) hipLaunchKernelGGL((store_kv_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((store_kv_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (fp8) hipLaunchKernelGGL((store_kv_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((store_kv_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_store_kv_rope(const RopeParams& p, int64_t n_units, int head_dim, bool fp8, bool interleaved,
                                hipStream_t stream) {
  if (n_units <= 0) return hipSuccess;
  dim3 grid((unsigned)n_units), block(kStoreThreads);
#define KVX_ROPE_LAUNCH(D, F, I) hipLaunchKernelGGL((store_kv_rope_kernel<D, F, I>), grid, block, 0, stream, p)
  if (head_dim == 128) {
    if (fp8) { if (interleaved) KVX_ROPE_LAUNCH(128, true, true); else KVX_ROPE_LAUNCH(128, true, false); }
    else { if (interleaved) KVX_ROPE_LAUNCH(128, false, true); else KVX_ROPE_LAUNCH(128, false, false); }
  } else {
    if (fp8) { if (interleaved) KVX_ROPE_LAUNCH(64, true, true); else KVX_ROPE_LAUNCH(64, true, false); }
    else { if (interleaved) KVX_ROPE_LAUNCH(64, false, true); else KVX_ROPE_LAUNCH(64, false, false); }
  }
#undef KVX_ROPE_LAUNCH
  return hipGetLastError();
}

hipError_t launch_page_move(const PageMoveParams& p, int64_t n_pages, hipStream_t stream) {
  if (n_pages <= 0) return hipSuccess;
  hipLaunchKernelGGL(page_move_kernel, dim3((unsigned)n_pages, 2), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_page_io(const PageIoParams& p, int64_t n_pages, int head_dim, int elem_bytes,
                          hipStream_t stream) {
  if (n_pages <= 0) return hipSuccess;
  dim3 grid((unsigned)n_pages, (unsigned)p.num_kv_heads), block(256);
  if (head_dim == 128) {
    if (elem_bytes == 2) hipLaunchKernelGGL((page_io_kernel<128, 2>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((page_io_kernel<128, 1>), grid, block, 0, stream, p);
  } else {
    if (elem_bytes == 2) hipLaunchKernelGGL((page_io_kernel<64, 2>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((page_io_kernel<64, 1>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace kvx
