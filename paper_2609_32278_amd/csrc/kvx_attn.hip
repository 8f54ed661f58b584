// Prefix-extend attention over a paged KV pool, gfx950 (CDNA4).
//
// Each suffix query at absolute position t of a request attends over keys
// 0..t of the request's logical sequence: the KV pages its cached prefix still
// holds, then the suffix itself, causally (the computation prefix caching
// reduces to the uncached suffix, paper Sections 1 and 2).
//
// Workgroup = 4 waves = one AttnUnit: 128 query rows (tile_tok suffix tokens x
// the `group` query heads that share one KV head) against a range of keys.
// Per 64-key tile:
//   * K [64 keys][D] and V^T [D][64 keys] pages are gathered through the page
//     table into LDS (double buffered; the next tile's global loads are issued
//     before the current tile's math);
//   * S^T = K * Q^T on v_mfma_f32_32x32x16_bf16: K rows are the A operand (read
//     from LDS), the wave's 32 query rows are the B operand (held in registers
//     for the whole unit).  In the result each lane owns one query row and 16
//     keys of it, so softmax statistics are per lane plus one exchange with the
//     other half of the wave (v_permlane32_swap);
//   * online softmax in base 2 with the running maximum moved only when a row's
//     maximum grows by more than 2^8 (values stay <= 2^8, the final division
//     cancels the reference point);
//   * O^T += V^T * P^T: V^T from LDS is the A operand, the probabilities stay in
//     registers as the B operand, converted to bf16 pairs.
// MFMA row m of the S^T product is assigned key perm(m) (bits 2 and 3 of m
// swapped), which makes the keys a lane holds in the S^T accumulators exactly
// the 8 consecutive keys its B operand slot needs in the P^T * V product.

#include "kvx_internal.h"

namespace kvx {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleThreshold = 8.0f;  // log2 units

__device__ __forceinline__ float pair_max(float x) {
  // v_permlane32_swap(x, x): r[0] holds the low half's value, r[1] the high half's,
  // in every lane, so the combination is identical in lanes l and l ^ 32.
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Key (within a 32-key block) held by MFMA row m of the S^T product.
__device__ __forceinline__ int row_key(int m) {
  return (m & 0x13) | ((m & 0x4) << 1) | ((m & 0x8) >> 1);
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

// 8 fp8 e4m3 codes -> 8 bf16 (exact: every e4m3 value is a bf16 value)
__device__ __forceinline__ uint4 fp8x8_to_bf16x8(uint2 c) {
  uint4 r;
  auto f0 = __builtin_amdgcn_cvt_pk_f32_fp8(c.x, false);
  auto f1 = __builtin_amdgcn_cvt_pk_f32_fp8(c.x, true);
  auto f2 = __builtin_amdgcn_cvt_pk_f32_fp8(c.y, false);
  auto f3 = __builtin_amdgcn_cvt_pk_f32_fp8(c.y, true);
  r.x = pack_bf16(f0[0], f0[1]);
  r.y = pack_bf16(f1[0], f1[1]);
  r.z = pack_bf16(f2[0], f2[1]);
  r.w = pack_bf16(f3[0], f3[1]);
  return r;
}

template <int D, bool FP8>
struct TileGeom {
  static constexpr int BN = kTileKeys;
  static constexpr int PAGES = BN / kPageSize;          // 4 pages per tile
  static constexpr int K_LD = D + 8;                    // padded LDS row strides (elements)
  static constexpr int V_LD = BN + 8;
  static constexpr int K_TILE = BN * K_LD;
  static constexpr int V_TILE = D * V_LD;
  static constexpr int STAGE = K_TILE + V_TILE;         // one buffer, elements
  static constexpr int CHUNKS = PAGES * 2 * D;          // 8-element chunks per tile, per K and per V
  static constexpr int PER_THREAD = CHUNKS / kAttnThreads;
  static_assert(CHUNKS % kAttnThreads == 0, "tile chunks must spread evenly");
};

// Global -> register prefetch of one K tile and one V^T tile.
template <int D, bool FP8>
struct TileRegs {
  using G = TileGeom<D, FP8>;
  uint4 k[G::PER_THREAD];
  uint4 v[G::PER_THREAD];
};

template <int D, bool FP8>
__device__ __forceinline__ void load_tile(TileRegs<D, FP8>& r, const AttnParams& p, const AttnUnit& u,
                                          int kv_head, int k0) {
  using G = TileGeom<D, FP8>;
  constexpr int EB = FP8 ? 1 : 2;  // bytes per pool element
  const int lp0 = k0 / kPageSize;
  int pid[G::PAGES];
#pragma unroll
  for (int j = 0; j < G::PAGES; j++) {
    const bool valid = (lp0 + j) * kPageSize < u.key_end;
    pid[j] = valid ? __builtin_amdgcn_readfirstlane(p.page_ids[u.page_base + lp0 + j]) : -1;
  }
  const bool tail = k0 + G::BN > u.key_end;
#pragma unroll
  for (int it = 0; it < G::PER_THREAD; it++) {
    const int c = threadIdx.x + it * kAttnThreads;
    const int j = c / (2 * D);       // page within the tile
    const int w = c % (2 * D);
    const int page = pid[j];
    // K chunk: slot w / (D/8), elements (w % (D/8)) * 8 .. +8
    const int ks = w / (D / 8), kc = w % (D / 8);
    // V^T chunk: dim row w / 2, slots (w % 2) * 8 .. +8
    const int vd = w / 2, vh = w % 2;
    uint4 kx = make_uint4(0, 0, 0, 0), vx = make_uint4(0, 0, 0, 0);
    if (page >= 0) {
      const size_t blk = ((size_t)page * p.num_kv_heads + kv_head) * (size_t)(kPageSize * D);
      const char* kb = (const char*)p.k_pool + (blk + (size_t)ks * D + kc * 8) * EB;
      const char* vb = (const char*)p.v_pool + (blk + (size_t)vd * kPageSize + vh * 8) * EB;
      if constexpr (FP8) {
        kx = fp8x8_to_bf16x8(*(const uint2*)kb);
        vx = fp8x8_to_bf16x8(*(const uint2*)vb);
      } else {
        kx = *(const uint4*)kb;
        vx = *(const uint4*)vb;
      }
      if (tail) {
        // keys at or beyond key_end are never weighted; zero them so that slots
        // never written (possibly NaN) cannot leak through 0 * NaN
        const int key_k = k0 + j * kPageSize + ks;
        if (key_k >= u.key_end) kx = make_uint4(0, 0, 0, 0);
        const int key_v = k0 + j * kPageSize + vh * 8;
        uint32_t* vw = (uint32_t*)&vx;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const uint32_t lo = (key_v + 2 * e < u.key_end) ? 0xFFFFu : 0u;
          const uint32_t hi = (key_v + 2 * e + 1 < u.key_end) ? 0xFFFF0000u : 0u;
          vw[e] &= (lo | hi);
        }
      }
    }
    r.k[it] = kx;
    r.v[it] = vx;
  }
}

template <int D, bool FP8>
__device__ __forceinline__ void store_tile(const TileRegs<D, FP8>& r, uint16_t* stage) {
  using G = TileGeom<D, FP8>;
  uint16_t* kt = stage;
  uint16_t* vt = stage + G::K_TILE;
#pragma unroll
  for (int it = 0; it < G::PER_THREAD; it++) {
    const int c = threadIdx.x + it * kAttnThreads;
    const int j = c / (2 * D);
    const int w = c % (2 * D);
    const int ks = w / (D / 8), kc = w % (D / 8);
    const int vd = w / 2, vh = w % 2;
    *(uint4*)(kt + (j * kPageSize + ks) * G::K_LD + kc * 8) = r.k[it];
    *(uint4*)(vt + vd * G::V_LD + j * kPageSize + vh * 8) = r.v[it];
  }
}

template <int D, bool FP8>
__global__ __launch_bounds__(kAttnThreads, 2) void extend_attn_kernel(AttnParams p) {
  using G = TileGeom<D, FP8>;
  constexpr int KSTEPS = D / 16;  // MFMA k-steps over head_dim
  constexpr int DB = D / 32;      // 32-wide blocks of head_dim in O^T
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * G::STAGE];

  const AttnUnit u = p.units[blockIdx.x];
  if (u.key_end <= u.key_begin) return;  // padding entry: uniform exit

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n = lane & 31;  // query row within the wave / MFMA row
  const int h = lane >> 5;  // half of the wave
  const int kv_head = u.head_ntok >> 16;
  const int ntok = u.head_ntok & 0xFFFF;

  // this lane's query row: row rho = token * group + head-in-group
  const int rho = wave * 32 + n;
  const int tok = rho / p.group;
  const int hq = kv_head * p.group + (rho - tok * p.group);
  const bool row_valid = tok < ntok;
  const int qpos = u.q_pos0 + tok;

  // Q^T operand: k-slot (h, j) of k-step s holds dim h*D/2 + 8s + j
  bf16x8 qf[KSTEPS];
  {
    const uint4* src = (const uint4*)(p.q + ((size_t)(u.qo_row0 + tok) * p.num_q_heads + hq) * D + h * (D / 2));
#pragma unroll
    for (int s = 0; s < KSTEPS; s++) {
      uint4 v = row_valid ? src[s] : make_uint4(0, 0, 0, 0);
      qf[s] = __builtin_bit_cast(bf16x8, v);
    }
  }

  float scale = p.scale_log2;
  float vscale = 1.0f;
  if constexpr (FP8) {
    scale *= p.k_scale[kv_head];
    vscale = p.v_scale[kv_head];
  }

  f32x16 o[DB];
#pragma unroll
  for (int b = 0; b < DB; b++) o[b] = f32x16{};
  float m_run = -1e30f;
  float l_run = 0.0f;

  const int k_first = u.key_begin;
  const int n_tiles = (u.key_end - k_first + G::BN - 1) / G::BN;
  const int krow0 = row_key(n);

  TileRegs<D, FP8> regs;
  load_tile<D, FP8>(regs, p, u, kv_head, k_first);
  store_tile<D, FP8>(regs, lds);
  __syncthreads();

  for (int t = 0; t < n_tiles; t++) {
    const int k0 = k_first + t * G::BN;
    const bool more = t + 1 < n_tiles;
    if (more) load_tile<D, FP8>(regs, p, u, kv_head, k0 + G::BN);

    const uint16_t* kt = lds + (t & 1) * G::STAGE;
    const uint16_t* vt = kt + G::K_TILE;

    // ---- S^T = K Q^T for two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int blk = 0; blk < 2; blk++) {
      s[blk] = f32x16{};
      const uint16_t* krow = kt + (blk * 32 + krow0) * G::K_LD + h * (D / 2);
#pragma unroll
      for (int st = 0; st < KSTEPS; st++) {
        bf16x8 a = *(const bf16x8*)(krow + st * 8);
        s[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], s[blk], 0, 0, 0);
      }
    }

    // ---- online softmax (base 2); accumulator i of block blk holds key
    //      k0 + 32*blk + 16*(i/8) + 8*h + i%8 of this lane's query row
    const bool masked = k0 + G::BN - 1 > u.q_pos0;
    float mx = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; blk++) {
#pragma unroll
      for (int i = 0; i < 16; i++) {
        float x = s[blk][i] * scale;
        if (masked) {
          const int key = k0 + blk * 32 + 16 * (i / 8) + 8 * h + (i % 8);
          x = key > qpos ? -INFINITY : x;
        }
        s[blk][i] = x;
        mx = fmaxf(mx, x);
      }
    }
    mx = pair_max(mx);
    if (__any(mx > m_run + kRescaleThreshold)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < DB; b++) o[b] *= alpha;
      m_run = m_new;
    }
    float rs = 0.0f;
#pragma unroll
    for (int blk = 0; blk < 2; blk++) {
#pragma unroll
      for (int i = 0; i < 16; i++) {
        const float e = __builtin_amdgcn_exp2f(s[blk][i] - m_run);
        s[blk][i] = e;
        rs += e;
      }
    }
    l_run += rs;

    // ---- O^T += V^T P^T, 16 keys per MFMA
#pragma unroll
    for (int blk = 0; blk < 2; blk++) {
#pragma unroll
      for (int hf = 0; hf < 2; hf++) {
        uint4 pw;
        pw.x = pack_bf16(s[blk][8 * hf + 0], s[blk][8 * hf + 1]);
        pw.y = pack_bf16(s[blk][8 * hf + 2], s[blk][8 * hf + 3]);
        pw.z = pack_bf16(s[blk][8 * hf + 4], s[blk][8 * hf + 5]);
        pw.w = pack_bf16(s[blk][8 * hf + 6], s[blk][8 * hf + 7]);
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
        const uint16_t* vrow = vt + n * G::V_LD + blk * 32 + 16 * hf + 8 * h;
#pragma unroll
        for (int b = 0; b < DB; b++) {
          bf16x8 a = *(const bf16x8*)(vrow + b * 32 * G::V_LD);
          o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[b], 0, 0, 0);
        }
      }
    }

    if (more) store_tile<D, FP8>(regs, lds + ((t + 1) & 1) * G::STAGE);
    __syncthreads();
  }

  // ---- epilogue: lane (n, h) holds dims 32*b + 8*(i/4) + 4*h + i%4 of its row
  const float l_tot = pair_sum(l_run);
  const float inv = l_tot > 0.0f ? vscale / l_tot : 0.0f;
  const float lse_val = l_tot > 0.0f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  if (u.part < 0) {
    if (row_valid) {
      uint16_t* dst = p.out + ((size_t)(u.qo_row0 + tok) * p.num_q_heads + hq) * D;
#pragma unroll
      for (int b = 0; b < DB; b++) {
#pragma unroll
        for (int g4 = 0; g4 < 4; g4++) {
          uint2 w;
          w.x = pack_bf16(o[b][4 * g4 + 0] * inv, o[b][4 * g4 + 1] * inv);
          w.y = pack_bf16(o[b][4 * g4 + 2] * inv, o[b][4 * g4 + 3] * inv);
          *(uint2*)(dst + 32 * b + 8 * g4 + 4 * h) = w;
        }
      }
      if (p.lse != nullptr && h == 0) p.lse[(size_t)(u.qo_row0 + tok) * p.num_q_heads + hq] = lse_val;
    }
  } else {
    float* dst = p.o_part + ((size_t)u.part * kTileRows + rho) * D;
#pragma unroll
    for (int b = 0; b < DB; b++) {
#pragma unroll
      for (int g4 = 0; g4 < 4; g4++) {
        f32x4 w;
        w[0] = o[b][4 * g4 + 0] * inv;
        w[1] = o[b][4 * g4 + 1] * inv;
        w[2] = o[b][4 * g4 + 2] * inv;
        w[3] = o[b][4 * g4 + 3] * inv;
        *(f32x4*)(dst + 32 * b + 8 * g4 + 4 * h) = w;
      }
    }
    if (h == 0) p.lse_part[(size_t)u.part * kTileRows + rho] = lse_val;
  }
}

// Combine the parts of split tiles: o = sum_p e^{lse_p - M} o_p / sum_p e^{lse_p - M}.
template <int D>
__global__ __launch_bounds__(256) void merge_kernel(MergeParams p) {
  const MergeUnit mu = p.merges[blockIdx.x];
  const int kv_head = mu.head_ntok >> 16;
  const int ntok = mu.head_ntok & 0xFFFF;
  constexpr int C4 = D / 4;
  for (int idx = threadIdx.x; idx < kTileRows * C4; idx += blockDim.x) {
    const int rho = idx / C4;
    const int c = (idx % C4) * 4;
    const int tok = rho / p.group;
    if (tok >= ntok) continue;
    const int hq = kv_head * p.group + (rho - tok * p.group);
    float mx = -INFINITY;
    for (int q = 0; q < mu.nparts; q++) mx = fmaxf(mx, p.lse_part[(size_t)(mu.part0 + q) * kTileRows + rho]);
    float wsum = 0.0f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int q = 0; q < mu.nparts; q++) {
      const float l = p.lse_part[(size_t)(mu.part0 + q) * kTileRows + rho];
      const float w = (l == -INFINITY) ? 0.0f : __expf(l - mx);
      const f32x4 v = *(const f32x4*)(p.o_part + ((size_t)(mu.part0 + q) * kTileRows + rho) * D + c);
      acc += v * w;
      wsum += w;
    }
    const float inv = wsum > 0.0f ? 1.0f / wsum : 0.0f;
    const size_t row = (size_t)(mu.qo_row0 + tok) * p.num_q_heads + hq;
    uint2 w2;
    w2.x = pack_bf16(acc[0] * inv, acc[1] * inv);
    w2.y = pack_bf16(acc[2] * inv, acc[3] * inv);
    *(uint2*)(p.out + row * D + c) = w2;
    if (p.lse != nullptr && c == 0) p.lse[row] = mx + __logf(wsum);
  }
}

}  // namespace

hipError_t launch_extend_attention(const AttnParams& p, int64_t n_units, int head_dim, bool fp8,
                                   hipStream_t stream) {
  if (n_units <= 0) return hipSuccess;
  dim3 grid((unsigned)n_units), block(kAttnThreads);
  if (head_dim == 128) {
    if (fp8) hipLaunchKernelGGL((extend_attn_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((extend_attn_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (fp8) hipLaunchKernelGGL((extend_attn_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((extend_attn_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_merge(const MergeParams& p, int64_t n_merges, int head_dim, hipStream_t stream) {
  if (n_merges <= 0) return hipSuccess;
  dim3 grid((unsigned)n_merges), block(256);
  if (head_dim == 128) hipLaunchKernelGGL((merge_kernel<128>), grid, block, 0, stream, p);
  else hipLaunchKernelGGL((merge_kernel<64>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace kvx
