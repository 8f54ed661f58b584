// Paged decode attention over the KV pool, gfx950 (CDNA4): one new token per
// request attends over the request's whole cached sequence (the decode step that
// follows prefill, paper Section 2 and Section 4's prefill-decode serving).
//
// A decode step reads every K/V byte of a request once for a handful of query
// rows (the G query heads of one KV head), so it is bound by HBM, not MFMA.  The
// kernel streams pages straight into registers with wide loads and keeps several
// page pairs in flight per wave:
//   * workgroup = one key chunk of one (request, KV head); 4 waves, wave w takes
//     page pairs w, w+4, w+8, ... of the chunk (two 16-key pages = 32 keys);
//   * S^T (16 keys x 16 rows) = K Q^T on v_mfma_f32_16x16x32_bf16: the page's keys
//     are the A operand straight from global memory, the G <= 16 query heads the B
//     operand (rows past G are zero);
//   * softmax in base 2, exact online rescaling (a row's four lane groups share
//     its running maximum through two lane swaps);
//   * O^T (16 dims x 16 rows per block) += V^T P^T, again 16x16x32: the 32 keys of
//     the pair are the reduction dimension, taken as key 4g..4g+3 of the first
//     page and of the second page in lane group g -- the keys that lane group
//     holds in the S^T result, so P needs no data movement between lanes;
//   * the four waves' partial results are combined through LDS; a chunk that is
//     one part of a split key range writes (O, LSE), merged afterwards.

#include <type_traits>

#include "kvx_internal.h"

namespace kvx {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;  // scalar-loaded

constexpr float kLn2 = 0.6931471805599453f;
constexpr int kWaves = kDecodeThreads / 64;
constexpr int kRows = kDecodeMaxGroup;

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

// max / sum over the four lane groups (lanes n, n+16, n+32, n+48) holding one row
__device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float group_sum(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// 8 fp8 e4m3 codes -> 8 bf16 and 4 codes -> 4 bf16 (exact: e4m3 values are bf16 values)
__device__ __forceinline__ uint4 fp8x8_bf16(uint2 c) {
  return make_uint4(__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.x, 1.0f, false)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.x, 1.0f, true)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.y, 1.0f, false)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.y, 1.0f, true)));
}
__device__ __forceinline__ uint2 fp8x4_bf16(uint32_t c) {
  return make_uint2(__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c, 1.0f, false)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c, 1.0f, true)));
}

// Registers of one page pair as loaded (fp8 pools: raw codes, converted when used).
template <int D, bool FP8>
struct PairRegs {
  using KT = typename std::conditional<FP8, uint2, uint4>::type;
  using VT = typename std::conditional<FP8, uint32_t, uint2>::type;
  KT ka[D / 32], kb[D / 32];  // K A-operands of the two pages, one per 32-dim step
  VT va[D / 16], vb[D / 16];  // V^T: slots 4g..4g+3 of each page, one per 16-dim block
};

template <int D, bool FP8>
__global__ __launch_bounds__(kDecodeThreads, 2) void decode_kernel(DecodeParams p) {
  constexpr int QS = D / 32;   // QK reduction steps
  constexpr int DB = D / 16;   // PV output blocks
  constexpr int PAGE_ELEMS = kPageSize * D;
  __shared__ float sm_m[kWaves][kRows], sm_l[kWaves][kRows];
  __shared__ float sm_o[kWaves][kRows][D];

  DecodeUnit u;
  {
    const const_i32_ptr w = (const_i32_ptr)(p.units + blockIdx.x);
    u.qo_row = w[0];
    u.page_base = w[1];
    u.key_begin = w[2];
    u.key_end = w[3];
    u.head = w[4];
    u.part = w[5];
  }
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15;   // A row (key within a page) / B, C column (query row)
  const int g = lane >> 4;   // lane group
  const int G = p.group;

  // Q^T B-operands: dims 32 s + 8 g .. +8 of query row n (zero past the group)
  bf16x8 qf[QS];
  {
    const bool valid = n < G;
    const uint4* src = (const uint4*)(p.q + ((size_t)u.qo_row * p.num_q_heads + u.head * G + (valid ? n : 0)) * D + 8 * g);
#pragma unroll
    for (int s = 0; s < QS; s++) qf[s] = __builtin_bit_cast(bf16x8, valid ? src[4 * s] : make_uint4(0, 0, 0, 0));
  }

  const size_t head_off = (size_t)u.head * PAGE_ELEMS;
  const size_t page_stride = (size_t)p.num_kv_heads * PAGE_ELEMS;
  const const_i32_ptr pages = (const_i32_ptr)p.page_ids + u.page_base;
  const int last_page = (u.key_end - 1) / kPageSize;
  const int lp0 = u.key_begin / kPageSize;
  const int n_pairs = (u.key_end - u.key_begin + 2 * kPageSize - 1) / (2 * kPageSize);

  using KT = typename PairRegs<D, FP8>::KT;
  using VT = typename PairRegs<D, FP8>::VT;
  constexpr int EB = FP8 ? 1 : 2;  // bytes per element
  // element offsets of the (page, KV head) blocks of pair `pair`; pages past the
  // end repeat the last one (their keys are masked)
  auto blocks = [&](int pair, size_t& pa, size_t& pb) {
    int la = lp0 + 2 * pair, lb = la + 1;
    la = la < last_page ? la : last_page;
    lb = lb < last_page ? lb : last_page;
    pa = (size_t)(uint32_t)pages[la] * page_stride + head_off;
    pb = (size_t)(uint32_t)pages[lb] * page_stride + head_off;
  };
  auto load_k = [&](size_t pa, size_t pb, PairRegs<D, FP8>& r) {
    const char* k = (const char*)p.k_pool;
#pragma unroll
    for (int s = 0; s < QS; s++) {
      r.ka[s] = *(const KT*)(k + (pa + n * D + 32 * s + 8 * g) * EB);
      r.kb[s] = *(const KT*)(k + (pb + n * D + 32 * s + 8 * g) * EB);
    }
  };
  auto load_v = [&](size_t pa, size_t pb, PairRegs<D, FP8>& r) {
    const char* v = (const char*)p.v_pool;
#pragma unroll
    for (int b = 0; b < DB; b++) {
      r.va[b] = *(const VT*)(v + (pa + (16 * b + n) * kPageSize + 4 * g) * EB);
      r.vb[b] = *(const VT*)(v + (pb + (16 * b + n) * kPageSize + 4 * g) * EB);
    }
  };

  f32x4 o[DB];
#pragma unroll
  for (int b = 0; b < DB; b++) o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  float scale = p.scale_log2;
  float vscale = 1.0f;
  if constexpr (FP8) {
    scale *= p.k_scale[u.head];
    vscale = p.v_scale[u.head];
  }

  // Pair `pair` from r; the registers are refilled with pair `next` (if < n_pairs)
  // as soon as the products have read them, so the loads of the next pair are in
  // flight for the rest of this one.
  auto compute = [&](int pair, int next, PairRegs<D, FP8>& r) {
    size_t na = 0, nb = 0;
    const bool more = next < n_pairs;  // uniform
    if (more) blocks(next, na, nb);
    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < QS; s++) {
      uint4 ka, kb;
      if constexpr (FP8) {
        ka = fp8x8_bf16(r.ka[s]);
        kb = fp8x8_bf16(r.kb[s]);
      } else {
        ka = r.ka[s];
        kb = r.kb[s];
      }
      sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka), qf[s], sa, 0, 0, 0);
      sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kb), qf[s], sb, 0, 0, 0);
    }
    if (more) load_k(na, nb, r);
    uint2 va[DB], vb[DB];
#pragma unroll
    for (int b = 0; b < DB; b++) {
      if constexpr (FP8) {
        va[b] = fp8x4_bf16(r.va[b]);
        vb[b] = fp8x4_bf16(r.vb[b]);
      } else {
        va[b] = r.va[b];
        vb[b] = r.vb[b];
      }
    }
    if (more) load_v(na, nb, r);
    // keys of this lane: 4g + i of page a (key0) and of page b (key0 + 16)
    const int key0 = u.key_begin + 32 * pair + 4 * g;
    const bool tail = u.key_begin + 32 * (pair + 1) > u.key_end;  // uniform
    if (tail) {
#pragma unroll
      for (int i = 0; i < 4; i++) {
        if (key0 + i >= u.key_end) sa[i] = -INFINITY;
        if (key0 + 16 + i >= u.key_end) sb[i] = -INFINITY;
      }
      // zero V of keys past the end: unwritten slots may hold NaN
      const uint32_t ma0 = (key0 + 0 < u.key_end ? 0xFFFFu : 0u) | (key0 + 1 < u.key_end ? 0xFFFF0000u : 0u);
      const uint32_t ma1 = (key0 + 2 < u.key_end ? 0xFFFFu : 0u) | (key0 + 3 < u.key_end ? 0xFFFF0000u : 0u);
      const uint32_t mb0 = (key0 + 16 < u.key_end ? 0xFFFFu : 0u) | (key0 + 17 < u.key_end ? 0xFFFF0000u : 0u);
      const uint32_t mb1 = (key0 + 18 < u.key_end ? 0xFFFFu : 0u) | (key0 + 19 < u.key_end ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int b = 0; b < DB; b++) {
        va[b].x &= ma0;
        va[b].y &= ma1;
        vb[b].x &= mb0;
        vb[b].y &= mb1;
      }
    }
    float mx = fmaxf(fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3])), fmaxf(fmaxf(sb[0], sb[1]), fmaxf(sb[2], sb[3])));
    mx = group_max(mx) * scale;
    if (__any(mx > m_run)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 when m_run = -inf
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < DB; b++) o[b] *= alpha;
      m_run = m_new;
    }
    // a row whose keys so far are all masked keeps m_run = -inf: its p are 0
    const float neg = m_run == -INFINITY ? 0.f : -m_run;
    float pa[4], pb[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      pa[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sa[i], scale, neg));
      pb[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sb[i], scale, neg));
    }
    const uint4 pw = make_uint4(pack2(pa[0], pa[1]), pack2(pa[2], pa[3]), pack2(pb[0], pb[1]), pack2(pb[2], pb[3]));
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.x), ones, l_run, false);
    l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.y), ones, l_run, false);
    l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.z), ones, l_run, false);
    l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.w), ones, l_run, false);
    const bf16x8 pbv = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int b = 0; b < DB; b++) {
      const uint4 vv = make_uint4(va[b].x, va[b].y, vb[b].x, vb[b].y);
      o[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vv), pbv, o[b], 0, 0, 0);
    }
  };

  PairRegs<D, FP8> r;
  if (wave < n_pairs) {
    size_t pa, pb;
    blocks(wave, pa, pb);
    load_k(pa, pb, r);
    load_v(pa, pb, r);
  }
  for (int j = wave; j < n_pairs; j += kWaves) compute(j, j + kWaves, r);

  // ---- combine the four waves.  Lane (n, g) holds dims 16 b + 4 g + i of row n.
  const float l_row = group_sum(l_run);
  if (g == 0) {
    sm_m[wave][n] = m_run;
    sm_l[wave][n] = l_row;
  }
#pragma unroll
  for (int b = 0; b < DB; b++)
#pragma unroll
    for (int i = 0; i < 4; i++) sm_o[wave][n][16 * b + 4 * g + i] = o[b][i];
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * D; idx += kDecodeThreads) {
    const int row = idx / D, d = idx - row * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; w++) M = fmaxf(M, sm_m[w][row]);
    float wsum = 0.f, acc = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; w++) {
        const float e = sm_m[w][row] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sm_m[w][row] - M);
        wsum += e * sm_l[w][row];
        acc += e * sm_o[w][row][d];
      }
    }
    const float val = wsum > 0.f ? acc * vscale / wsum : 0.f;
    const float lse_v = wsum > 0.f ? (M + __log2f(wsum)) * kLn2 : -INFINITY;
    if (u.part < 0) {
      const size_t orow = (size_t)u.qo_row * p.num_q_heads + u.head * G + row;
      p.out[orow * D + d] = __builtin_bit_cast(uint16_t, (__bf16)val);
      if (p.lse != nullptr && d == 0) p.lse[orow] = lse_v;
    } else {
      p.o_part[((size_t)u.part * kRows + row) * D + d] = val;
      if (d == 0) p.lse_part[(size_t)u.part * kRows + row] = lse_v;
    }
  }
}

// Combine the parts of a split decode key range: o = sum_p e^{lse_p - M} o_p / sum_p e^{lse_p - M}.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeMergeParams p) {
  const DecodeMerge mu = p.merges[blockIdx.x];
  const int G = p.group;
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int row = idx / D, d = idx - row * D;
    float M = -INFINITY;
    for (int q = 0; q < mu.nparts; q++) M = fmaxf(M, p.lse_part[(size_t)(mu.part0 + q) * kRows + row]);
    float wsum = 0.f, acc = 0.f;
    for (int q = 0; q < mu.nparts; q++) {
      const float l = p.lse_part[(size_t)(mu.part0 + q) * kRows + row];
      const float w = l == -INFINITY ? 0.f : __expf(l - M);
      wsum += w;
      acc += w * p.o_part[((size_t)(mu.part0 + q) * kRows + row) * D + d];
    }
    const size_t orow = (size_t)mu.qo_row * p.num_q_heads + mu.head * G + row;
    p.out[orow * D + d] = __builtin_bit_cast(uint16_t, (__bf16)(wsum > 0.f ? acc / wsum : 0.f));
    if (p.lse != nullptr && d == 0) p.lse[orow] = M + __logf(wsum);
  }
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, int64_t n_units, int head_dim, bool fp8, hipStream_t stream) {
  if (n_units <= 0) return hipSuccess;
  const dim3 grid((unsigned)n_units), block(kDecodeThreads);
  if (head_dim == 128) {
    if (fp8) hipLaunchKernelGGL((decode_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((decode_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (fp8) hipLaunchKernelGGL((decode_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((decode_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_decode_merge(const DecodeMergeParams& p, int64_t n_merges, int head_dim, hipStream_t stream) {
  if (n_merges <= 0) return hipSuccess;
  if (head_dim == 128) hipLaunchKernelGGL(decode_merge_kernel<128>, dim3((unsigned)n_merges), dim3(256), 0, stream, p);
  else hipLaunchKernelGGL(decode_merge_kernel<64>, dim3((unsigned)n_merges), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace kvx
