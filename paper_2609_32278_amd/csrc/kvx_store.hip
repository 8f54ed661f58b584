// KV store into the paged pool and raw page I/O, gfx950 (CDNA4).
//
// Prefill materialises the suffix's K/V in every attention layer (paper,
// Section 2); store_kv writes them into the request's pages so that the next
// attention pass -- and every later turn that reuses this prefix -- reads them
// from the pool.  HBM-bound: each element is read once and written once.
//
// Pool layout: K [page][kv_head][slot][dim], V [page][kv_head][dim][slot].
// One workgroup handles one page of one request (all KV heads): K rows are
// copied with 16-byte accesses, V rows are staged in LDS and written out
// transposed, one 16-slot column (32 bytes bf16 / 16 bytes fp8) per dim.
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

template <int D, bool FP8>
__global__ __launch_bounds__(kStoreThreads) void store_kv_kernel(StoreParams p) {
  // V rows of this page for one head, staged for the transpose: [16 slots][D] bf16
  __shared__ __attribute__((aligned(16))) uint16_t vs[kPageSize][D + 8];
  const StoreUnit su = p.units[blockIdx.x];
  const int page = p.page_ids[su.page_pos];
  const int H = p.num_kv_heads;
  constexpr int CPR = D / 8;                // 16-byte chunks per bf16 row
  constexpr int CHUNKS = kPageSize * CPR;   // per head
  const bool full = su.slot_begin == 0 && su.slot_end == kPageSize;

  for (int hd = 0; hd < H; hd++) {
    const float kinv = FP8 ? p.k_inv_scale[hd] : 1.0f;
    const float vinv = FP8 ? p.v_inv_scale[hd] : 1.0f;
    const size_t blk = ((size_t)page * H + hd) * (size_t)(kPageSize * D);
    for (int c = threadIdx.x; c < CHUNKS; c += kStoreThreads) {
      const int slot = c / CPR, cc = c % CPR;
      uint4 kx = make_uint4(0, 0, 0, 0), vx = make_uint4(0, 0, 0, 0);
      const bool live = slot >= su.slot_begin && slot < su.slot_end;
      if (live) {
        const size_t src = ((size_t)(su.row_slot0 + slot) * H + hd) * D + cc * 8;
        kx = *(const uint4*)(p.k_ext + src);
        vx = *(const uint4*)(p.v_ext + src);
        if constexpr (FP8) {
          const uint16_t* ke = (const uint16_t*)&kx;
          uint2 code;
          code.x = e4m3x4(bf16_to_f32(ke[0]) * kinv, bf16_to_f32(ke[1]) * kinv,
                          bf16_to_f32(ke[2]) * kinv, bf16_to_f32(ke[3]) * kinv);
          code.y = e4m3x4(bf16_to_f32(ke[4]) * kinv, bf16_to_f32(ke[5]) * kinv,
                          bf16_to_f32(ke[6]) * kinv, bf16_to_f32(ke[7]) * kinv);
          *(uint2*)((uint8_t*)p.k_pool + blk + (size_t)slot * D + cc * 8) = code;
        } else {
          *(uint4*)((uint16_t*)p.k_pool + blk + (size_t)slot * D + cc * 8) = kx;
        }
      }
      *(uint4*)(&vs[slot][cc * 8]) = vx;
    }
    __syncthreads();
    // V^T: dim d, slots [8*half, 8*half+8)
    for (int c = threadIdx.x; c < 2 * D; c += kStoreThreads) {
      const int d = c / 2, half = c % 2;
      const int s0 = half * 8;
      if (s0 + 8 <= su.slot_begin || s0 >= su.slot_end) continue;
      float x[8];
      uint16_t raw[8];
#pragma unroll
      for (int e = 0; e < 8; e++) {
        raw[e] = vs[s0 + e][d];
        x[e] = bf16_to_f32(raw[e]) * vinv;
      }
      const bool whole = full || (s0 >= su.slot_begin && s0 + 8 <= su.slot_end);
      if constexpr (FP8) {
        uint8_t* dst = (uint8_t*)p.v_pool + blk + (size_t)d * kPageSize + s0;
        uint2 code;
        code.x = e4m3x4(x[0], x[1], x[2], x[3]);
        code.y = e4m3x4(x[4], x[5], x[6], x[7]);
        if (whole) {
          *(uint2*)dst = code;
        } else {
          const uint8_t* cb = (const uint8_t*)&code;
          for (int e = 0; e < 8; e++)
            if (s0 + e >= su.slot_begin && s0 + e < su.slot_end) dst[e] = cb[e];
        }
      } else {
        uint16_t* dst = (uint16_t*)p.v_pool + blk + (size_t)d * kPageSize + s0;
        if (whole) {
          uint4 w;
          w.x = raw[0] | ((uint32_t)raw[1] << 16);
          w.y = raw[2] | ((uint32_t)raw[3] << 16);
          w.z = raw[4] | ((uint32_t)raw[5] << 16);
          w.w = raw[6] | ((uint32_t)raw[7] << 16);
          *(uint4*)dst = w;
        } else {
          for (int e = 0; e < 8; e++)
            if (s0 + e >= su.slot_begin && s0 + e < su.slot_end) dst[e] = raw[e];
        }
      }
    }
    __syncthreads();
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
  dim3 grid((unsigned)n_units), block(kStoreThreads);
  if (head_dim == 128) {
    if (fp8) hipLaunchKernelGGL((store_kv_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((store_kv_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (fp8) hipLaunchKernelGGL((store_kv_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((store_kv_kernel<64, false>), grid, block, 0, stream, p);
  }
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
