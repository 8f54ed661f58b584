// Prefix-extend attention over a paged KV pool, gfx950 (CDNA4).
//
// Each suffix query at absolute position t of a request attends over keys
// 0..t of the request's logical sequence: the KV pages its cached prefix still
// holds, then the suffix itself, causally (the computation prefix caching
// reduces to the uncached suffix, paper Sections 1 and 2).
//
// Workgroup = 8 waves = one AttnUnit: 256 query rows (tile_tok suffix tokens x
// the `group` query heads that share one KV head) against a range of keys, one
// workgroup per CU (two waves per SIMD).  Each wave owns 32 rows.
//
// Per 64-key tile t (four pages):
//   * K(t) and V^T(t) pages are gathered from the pool straight into LDS
//     (global_load_lds_dwordx4, no staging registers) through a 4-deep ring:
//     iteration t issues K(t+4) and V(t+3) -- one load per wave after every
//     quarter of the S(t+1) product, so the loads of a CU trickle into the
//     address units instead of arriving as one burst -- and waits only for the
//     loads issued two iterations earlier, so each load has three iterations to
//     arrive.  Page ids are read with scalar loads one iteration ahead, after the
//     iteration's last LDS operand read (an outstanding scalar load would make
//     every LDS wait a full drain).
//   * S^T(t) = K(t) Q^T on v_mfma_f32_32x32x16_bf16: K rows are the A operand
//     (LDS), the wave's query rows the B operand (registers for the whole unit).
//     In the result each lane owns one query row and 16 keys of it, so softmax
//     statistics are per lane plus one v_permlane32_swap;
//   * online softmax in base 2: p = exp2(s * scale - m) (one FMA + one exp per
//     score) against a reference point m that stays at the row maximum of the
//     unit's first tile: no per-tile maximum and no rescale in the loop (the
//     final division cancels m).  bf16 P and fp32 O and l keep their relative
//     precision for p far above 1, so this is exact unless a later score beats
//     the first tile's maximum by so much that an exponential or a sum overflows
//     fp32.  A workgroup whose results are not all finite therefore runs the
//     unit a second time with a moving reference (a row's maximum moves when it
//     grows by more than 2^8, with O and l rescaled).  Folded form (always on an
//     fp8 pool; on a bf16 pool when the pool's scaled-Q setting asks for it): the
//     FMA goes away.  Q is multiplied by scale (times k_scale on an fp8 pool)
//     when it is loaded and rounded once more to bf16 (2^-9 relative; on an fp8
//     pool far below the e4m3 rounding of K), and the first MFMA of every score
//     tile takes -m (a 16-register block) as its accumulator input, so the tile
//     comes out as s * scale - m and p is exp2 of it directly;
//   * O^T += V^T(t) P^T(t): V^T from LDS is the A operand, P stays in registers
//     as bf16 pairs, and the row sums are taken over those bf16 values (v_dot2).
// Software pipeline: the MFMAs of S(t+1) are issued among the exp / pack of tile
// t; the MFMAs of O += P(t) V(t) overlap, in the exact form's fixed-reference
// pass, the FMAs that turn S(t+1) into exponents, and in the second pass the row
// maximum of tile t+1.
// MFMA row m of the S^T product is assigned key perm(m) (bits 2 and 3 of m
// swapped), which makes the keys a lane holds in the S^T accumulators exactly
// the 8 consecutive keys its B operand slot needs in the V^T P^T product.

#include "kvx_internal.h"

namespace kvx {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;  // scalar-loaded

constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleThreshold = 8.0f;  // log2 units
constexpr int kWaves = kAttnThreads / 64;
constexpr int kKB = 2;        // 32-key MFMA blocks per LDS tile
constexpr int kBN = 32 * kKB; // keys per LDS tile; split boundaries are multiples of it
static_assert(kWaves * 32 == kTileRows, "one 32-row MFMA block per wave");
static_assert(kTileKeys % kBN == 0, "split boundaries must fall on tile boundaries");

// compile-time flags passed to the pipelined iteration
struct False { static constexpr bool value = false; };
struct True { static constexpr bool value = true; };
template <int N>
struct Stage { static constexpr int value = N; };  // ring slot of tile t, or -1: computed from t
using AnyStage = Stage<-1>;

__device__ __forceinline__ float pair_max(float x) {
  // v_permlane32_swap(x, x): r[0] holds the low half's value, r[1] the high half's,
  // in every lane, so the combination is identical in lanes l and l ^ 32.  The
  // inputs are scores (never signalling NaNs), so a plain v_max_f32 does, without
  // the canonicalising copies fmaxf would add.
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  float m;
  asm("v_max_f32 %0, %1, %2" : "=v"(m) : "v"(__uint_as_float(r[0])), "v"(__uint_as_float(r[1])));
  return m;
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
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

// 8 fp8 e4m3 codes -> 8 bf16, two per instruction with a unit scale (exact: every
// e4m3 value is a bf16 value)
__device__ __forceinline__ uint4 fp8x8_to_bf16x8(uint2 c) {
  uint4 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.x, 1.0f, false));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.x, 1.0f, true));
  r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.y, 1.0f, false));
  r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.y, 1.0f, true));
  return r;
}

template <int D>
struct Geom {
  static constexpr int KSTEPS = D / 16;          // MFMA k-steps over head_dim
  static constexpr int DB = D / 32;              // 32-wide head_dim blocks of O^T
  static constexpr int CPR = D / 8;              // 16-byte chunks per bf16 K row
  static constexpr int TILE_BYTES = kBN * D * 2; // bf16 K tile == bf16 V^T tile
  static constexpr int INSTR = TILE_BYTES / 1024;        // 1 KiB direct loads per tile (K or V)
  static constexpr int PER_WAVE = 2 * INSTR / kWaves;    // K and V loads of one wave per iteration
  static constexpr int K_SLOTS = INSTR / kWaves;         // slots [0, K_SLOTS) load K, the rest V^T
  static_assert(INSTR % kWaves == 0, "K and V loads must each spread evenly over waves");
  static constexpr int NSTAGE = 4;               // LDS ring depth for K and for V^T
  static_assert((2 * INSTR) % kWaves == 0, "loads must spread evenly over waves");
};

// LDS layouts (unpadded, XOR-swizzled so that the MFMA operand reads are free of
// bank conflicts while every 1 KiB of a tile can be written by one wave-wide
// direct load):
//   K tile   [kBN keys][D] bf16; 16-byte chunk c of key row r is stored at chunk
//            c ^ (r % CPR) of that row.
//   V^T tile [kBN/16 pages][D dims][16 slots] bf16; 16-byte chunk c (slots
//            8c..8c+7) of dim row d is stored at chunk c ^ ((d >> 3) & 1).
// Load g = it * 8 + wave of a tile pair is K load j = g (g < INSTR) or V load
// j = g - INSTR; lane l of load j writes bytes [1024 j + 16 l, +16) of its tile.
//   K: row r = j * (64 / CPR) + l / CPR, stored chunk l % CPR.
//   V: page j / (D/32), dim (j % (D/32)) * 32 + l / 2, stored chunk l % 2.
// Each load falls inside one page.

struct Ctx {
  const_i32_ptr page_ids;  // this request's page list
  const void* k_pool;
  const void* v_pool;
  int num_kv_heads;
  int page_base;
  int key_end;
  int kv_head;
};

// Physical page (uniform, scalar load) holding logical page lp of the unit's
// request; pages at or past key_end fall back to the page holding key_end - 1, so
// every address stays inside the pool (their keys are masked, and V is zeroed on
// the register path).
__device__ __forceinline__ int page_of(const Ctx& c, int lp) {
  const int last = (c.key_end - 1) / kPageSize;
  return c.page_ids[(uint32_t)(lp < last ? lp : last)];
}

template <int D>
struct LoadSlot {
  bool is_v;     // this slot loads V^T (else K)
  int j;         // load index within the tile
  int off;       // per-lane byte offset inside the page block (bf16 elements x 2)
  int page_sel;  // which page (0/1) of the tile
  __device__ __forceinline__ void init(int g, int lane) {
    using G = Geom<D>;
    is_v = g >= G::INSTR;
    j = is_v ? g - G::INSTR : g;
    if (is_v) {
      const int d = (j % (D / 32)) * 32 + lane / 2;
      const int ch = (lane % 2) ^ ((d >> 3) & 1);
      off = (d * kPageSize + ch * 8) * 2;
      page_sel = j / (D / 32);
    } else {
      const int r = j * (64 / G::CPR) + lane / G::CPR;
      const int ch = (lane % G::CPR) ^ (r % G::CPR);
      off = ((r % kPageSize) * D + ch * 8) * 2;
      page_sel = r / kPageSize;
    }
  }
};

// Byte address of (physical page, this unit's KV head) in the pool of the slot.
__device__ __forceinline__ const char* page_block(const char* head_base, uint32_t page, uint32_t page_bytes) {
  return head_base + (uint64_t)page * page_bytes;
}

// Direct global -> LDS load of one 1 KiB piece of a bf16 tile (no registers):
// lane l's 16 bytes at base + off land at LDS address lds + 16 l.  Issued as
// inline assembly so that the compiler's wait-count tracking, which cannot tell
// the ring slots apart and would drain every outstanding load before the next
// one and before each barrier, stays out of the way; the kernel orders these
// loads itself with explicit vmcnt waits and barriers.
__device__ __forceinline__ void lds_dma_16(const char* sbase, int voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2"
      :
      : "s"(lds), "v"(voff), "s"(sbase)
      : "memory", "m0");
}

template <int D>
__device__ __forceinline__ void issue_direct(const LoadSlot<D>& s, const char* block, uint8_t* tile) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)(tile + s.j * 1024);
  lds_dma_16(block, s.off, lds);
}

// Zero the bf16 V^T values of one piece whose keys lie at or past key_end (the
// piece holds slots elem % 16 .. +7 of page page_sel of the tile at key k0), so
// that unwritten, possibly NaN, slots never meet a zero weight.  Keys past key_end
// in K need nothing: their scores are masked.
template <int D>
__device__ __forceinline__ uint4 mask_v_tail(uint4 x, const LoadSlot<D>& s, int k0, int key_end) {
  const int key = k0 + s.page_sel * kPageSize + (s.off / 2) % kPageSize;
  uint32_t* xw = (uint32_t*)&x;
#pragma unroll
  for (int e = 0; e < 4; e++) {
    const uint32_t lo = (key + 2 * e < key_end) ? 0xFFFFu : 0u;
    const uint32_t hi = (key + 2 * e + 1 < key_end) ? 0xFFFF0000u : 0u;
    xw[e] &= (lo | hi);
  }
  return x;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  // s_waitcnt with only the vector-memory counter limited (expcnt, lgkmcnt at max)
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most `n` direct loads (the most recent ones) are outstanding.
template <int MAX, int N = MAX>
__device__ __forceinline__ void wait_issued(int n) {
  if constexpr (N == 0) {
    wait_vmcnt<0>();
  } else {
    if (n >= N) { wait_vmcnt<N>(); return; }
    wait_issued<MAX, N - 1>(n);
  }
}

// S^T of one tile for this wave's 32 rows: s[kb] holds keys 32 kb .. 32 kb + 31
// (the swizzle of a key row depends on the row modulo 16 only, so block kb reads
// at the same offsets shifted by 32 rows).
// between(i) runs after k-step group i of the PER_WAVE groups (used to spread
// this wave's loads of later tiles over the product).
// The first k-step accumulates onto c0: zero, or (folded softmax) the negated
// running maxima of the lanes' rows.
template <int D, typename F>
__device__ __forceinline__ void qk_tile(f32x16 (&s)[kKB], const uint8_t* kt, const int (&koff)[Geom<D>::KSTEPS],
                                        const bf16x8 (&qf)[Geom<D>::KSTEPS], const f32x16& c0, F&& between) {
  using G = Geom<D>;
  constexpr int STEP = G::KSTEPS / G::PER_WAVE;
#pragma unroll
  for (int st = 0; st < G::KSTEPS; st++) {
#pragma unroll
    for (int kb = 0; kb < kKB; kb++) {
      const bf16x8 a = *(const bf16x8*)(kt + kb * 32 * D * 2 + koff[st]);
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], st == 0 ? c0 : s[kb], 0, 0, 0);
    }
    if ((st + 1) % STEP == 0) between((st + 1) / STEP - 1);
  }
}

template <int D>
__device__ __forceinline__ void qk_tile(f32x16 (&s)[kKB], const uint8_t* kt, const int (&koff)[Geom<D>::KSTEPS],
                                        const bf16x8 (&qf)[Geom<D>::KSTEPS], const f32x16& c0) {
  qk_tile<D>(s, kt, koff, qf, c0, [](int) {});
}

// Raw row maximum of a tile (optionally causally masked in place), combined over
// both halves of the wave.  Accumulator i of block kb holds key
// k0 + 32 kb + 16 (i/8) + 8 h + i%8.
template <bool MASK>
__device__ __forceinline__ float row_max(f32x16 (&s)[kKB], int k0, int qpos, int h) {
  float m = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < kKB; kb++) {
#pragma unroll
    for (int i = 0; i < 16; i++) {
      float x = s[kb][i];
      if constexpr (MASK) {
        const int key = k0 + 32 * kb + 16 * (i / 8) + 8 * h + (i % 8);
        x = key > qpos ? -INFINITY : x;
        s[kb][i] = x;
      }
      m = fmaxf(m, x);
    }
  }
  return pair_max(m);
}

// Causal mask of a tile in place (keys past the row's position become -inf).
__device__ __forceinline__ void causal_mask(f32x16 (&s)[kKB], int k0, int qpos, int h) {
#pragma unroll
  for (int kb = 0; kb < kKB; kb++) {
#pragma unroll
    for (int i = 0; i < 16; i++) {
      const int key = k0 + 32 * kb + 16 * (i / 8) + 8 * h + (i % 8);
      s[kb][i] = key > qpos ? -INFINITY : s[kb][i];
    }
  }
}

// Whether a lane's results are finite (inf and NaN propagate through the sum; an
// overflow of the sum itself only reports a false alarm).
template <int D>
__device__ __forceinline__ bool all_finite(const f32x16 (&o)[Geom<D>::DB], float l) {
  float acc = l;
#pragma unroll
  for (int b = 0; b < Geom<D>::DB; b++)
#pragma unroll
    for (int i = 0; i < 16; i++) acc += o[b][i];
  return __builtin_isfinite(acc);
}

// s * scale - m in place (the exponent of the exact form), exactly as exp_pack forms it.
__device__ __forceinline__ void prescale(f32x16 (&s)[kKB], float scale, float m_run) {
  const float neg = -m_run;
#pragma unroll
  for (int kb = 0; kb < kKB; kb++)
#pragma unroll
    for (int i = 0; i < 16; i++) s[kb][i] = __builtin_fmaf(s[kb][i], scale, neg);
}

// p = exp2(s * scale - m) as bf16 pairs (the P^T B operands, one per page of the
// tile); returns the row sum over those bf16 values added to l.
// FOLDED: the tile is already s * scale - m, and p = exp2 of it.
template <bool FOLDED>
__device__ __forceinline__ float exp_pack(const f32x16 (&s)[kKB], bf16x8 (&pb)[2 * kKB], float l, float m_run,
                                          float scale) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  const float neg = -m_run;
  auto arg = [&](float x) { return FOLDED ? x : __builtin_fmaf(x, scale, neg); };
#pragma unroll
  for (int pg = 0; pg < 2 * kKB; pg++) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; e++) {
      const float p0 = __builtin_amdgcn_exp2f(arg(s[pg / 2][8 * (pg % 2) + 2 * e]));
      const float p1 = __builtin_amdgcn_exp2f(arg(s[pg / 2][8 * (pg % 2) + 2 * e + 1]));
      w[e] = pack_bf16(p0, p1);
      l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, l, false);
    }
    pb[pg] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
  }
  return l;
}

// O^T += V^T P^T: page pg of the tile against keys 16 pg .. 16 pg + 15.
template <int D>
__device__ __forceinline__ void pv_tile(f32x16 (&o)[Geom<D>::DB], const uint8_t* vt, int vbase,
                                        const bf16x8 (&pb)[2 * kKB]) {
  using G = Geom<D>;
#pragma unroll
  for (int pg = 0; pg < 2 * kKB; pg++) {
#pragma unroll
    for (int b = 0; b < G::DB; b++) {
      const bf16x8 a = *(const bf16x8*)(vt + pg * (D * 32) + b * 1024 + vbase);
      o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[pg], o[b], 0, 0, 0);
    }
  }
}

// ---------------------------------------------------------------- shared by both kernels

// Folded online softmax state of a lane's row, in log2 units of the scaled scores:
// the reference point m, the row sum l relative to it, -m as a 16-register
// accumulator input of every score tile's first k-step, and mx, the maximum of the
// newest tile relative to m.

// After the first tile: m = its row maximum (finite, because the unit's first key is
// visible to every row of the unit), and that tile is moved to it.
__device__ __forceinline__ void set_reference(f32x16 (&s)[kKB], float& mx, float& m_run, f32x16& cneg) {
  m_run = mx;
#pragma unroll
  for (int kb = 0; kb < kKB; kb++) s[kb] -= mx;
  cneg = -mx;
  mx = 0.0f;
}

// Lazy rescale before the tile st (maximum mx) is exponentiated: m moves only when a
// row outgrows it by 2^8 (kRescaleThreshold), and O, l and st move with it.
template <int D>
__device__ __forceinline__ void folded_rescale(f32x16 (&st)[kKB], f32x16 (&o)[Geom<D>::DB], float& mx, float& m_run,
                                               float& l_run, f32x16& cneg) {
  if (__any(mx > kRescaleThreshold)) {
    const float d = fmaxf(mx, 0.0f);
    const float alpha = __builtin_amdgcn_exp2f(-d);
    l_run *= alpha;
#pragma unroll
    for (int b = 0; b < Geom<D>::DB; b++) o[b] *= alpha;
#pragma unroll
    for (int kb = 0; kb < kKB; kb++) st[kb] -= d;
    m_run += d;
    mx -= d;
    cneg = -m_run;
  }
}

// The work item of this workgroup (scalar loads: every index derived from it stays
// uniform) and the lane's query row within it.
struct Rows {
  AttnUnit u;
  int lane, wave;
  int n;        // query row within the wave's block / MFMA row
  int h;        // half of the wave
  int kv_head, ntok;
  int rho;      // row of the unit: token * group + head-in-group
  int tok, hq, qpos;
  bool valid;   // the row is a real query (its token exists)
};

__device__ __forceinline__ Rows rows_of(const AttnParams& p) {
  Rows r;
  const const_i32_ptr w = (const_i32_ptr)(p.units + blockIdx.x);
  r.u.qo_row0 = w[0];
  r.u.q_pos0 = w[1];
  r.u.page_base = w[2];
  r.u.key_begin = w[3];
  r.u.key_end = w[4];
  r.u.head_ntok = w[5];
  r.u.part = w[6];
  r.u.req = w[7];
  r.lane = threadIdx.x & 63;
  r.wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  r.n = r.lane & 31;
  r.h = r.lane >> 5;
  r.kv_head = r.u.head_ntok >> 16;
  r.ntok = r.u.head_ntok & 0xFFFF;
  r.rho = r.wave * 32 + r.n;
  r.tok = r.rho / p.group;
  r.hq = r.kv_head * p.group + (r.rho - r.tok * p.group);
  r.valid = r.tok < r.ntok;
  r.qpos = r.u.q_pos0 + r.tok;
  return r;
}

// Q^T operand: k-slot (h, j) of k-step s holds dim h*D/2 + 8s + j.  SCALED: times
// `scale`, rounded once to bf16.
template <int D, bool SCALED>
__device__ __forceinline__ void load_q(bf16x8 (&qf)[Geom<D>::KSTEPS], const AttnParams& p, const Rows& r,
                                       float scale) {
  const uint4* src = (const uint4*)(p.q + ((size_t)(r.u.qo_row0 + r.tok) * p.num_q_heads + r.hq) * D + r.h * (D / 2));
#pragma unroll
  for (int s = 0; s < Geom<D>::KSTEPS; s++) {
    const uint4 raw = r.valid ? src[s] : make_uint4(0, 0, 0, 0);
    if constexpr (SCALED) {
      const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
      uint32_t o4[4];
#pragma unroll
      for (int e = 0; e < 4; e++)
        o4[e] = pack_bf16(__uint_as_float(w[e] << 16) * scale, __uint_as_float(w[e] & 0xFFFF0000u) * scale);
      qf[s] = __builtin_bit_cast(bf16x8, make_uint4(o4[0], o4[1], o4[2], o4[3]));
    } else {
      qf[s] = __builtin_bit_cast(bf16x8, raw);
    }
  }
}

// LDS read offsets of the MFMA operands.  K: MFMA row n holds key row_key(n); k-step
// st reads dims h*D/2 + 8st .. +8, i.e. chunk h*CPR/2 + st, stored swizzled.
template <int D>
__device__ __forceinline__ void k_offsets(int (&koff)[Geom<D>::KSTEPS], int n, int h) {
  const int r = row_key(n);
#pragma unroll
  for (int st = 0; st < Geom<D>::KSTEPS; st++)
    koff[st] = r * (D * 2) + (((h * (Geom<D>::CPR / 2) + st) ^ (r % Geom<D>::CPR)) * 16);
}

// V^T: dim 32b + n, slots 8h..8h+7 of a page.
__device__ __forceinline__ int v_offset(int n, int h) { return n * 32 + ((h ^ ((n >> 3) & 1)) * 16); }

// Epilogue: lane (n, h) holds dims 32*b + 8*(i/4) + 4*h + i%4 of its row; O = o * vscale / l
// rounded to bf16 with the LSE, or the fp32 partial result of a split part.
template <int D>
__device__ __forceinline__ void write_result(const AttnParams& p, const Rows& r, const f32x16 (&o)[Geom<D>::DB],
                                             float l_run, float m_run, float vscale) {
  using G = Geom<D>;
  const float l_tot = pair_sum(l_run);
  const float inv = l_tot > 0.0f ? vscale / l_tot : 0.0f;
  const float lse_val = l_tot > 0.0f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  if (r.u.part < 0) {
    if (r.valid) {
      uint16_t* dst = p.out + ((size_t)(r.u.qo_row0 + r.tok) * p.num_q_heads + r.hq) * D;
#pragma unroll
      for (int b = 0; b < G::DB; b++) {
#pragma unroll
        for (int g4 = 0; g4 < 4; g4++) {
          uint2 w;
          w.x = pack_bf16(o[b][4 * g4 + 0] * inv, o[b][4 * g4 + 1] * inv);
          w.y = pack_bf16(o[b][4 * g4 + 2] * inv, o[b][4 * g4 + 3] * inv);
          *(uint2*)(dst + 32 * b + 8 * g4 + 4 * r.h) = w;
        }
      }
      if (p.lse != nullptr && r.h == 0) p.lse[(size_t)(r.u.qo_row0 + r.tok) * p.num_q_heads + r.hq] = lse_val;
    }
  } else {
    float* dst = p.o_part + ((size_t)r.u.part * kTileRows + r.rho) * D;
#pragma unroll
    for (int b = 0; b < G::DB; b++) {
#pragma unroll
      for (int g4 = 0; g4 < 4; g4++) {
        f32x4 w;
        w[0] = o[b][4 * g4 + 0] * inv;
        w[1] = o[b][4 * g4 + 1] * inv;
        w[2] = o[b][4 * g4 + 2] * inv;
        w[3] = o[b][4 * g4 + 3] * inv;
        *(f32x4*)(dst + 32 * b + 8 * g4 + 4 * r.h) = w;
      }
    }
    if (r.h == 0) p.lse_part[(size_t)r.u.part * kTileRows + r.rho] = lse_val;
  }
}

// ---------------------------------------------------------------- bf16 pool

// SQ: folded softmax (Q scaled and rounded once more to bf16, see the file header).
template <int D, bool SQ>
__global__ __launch_bounds__(kAttnThreads, 1) void extend_attn_kernel(AttnParams p) {
  using G = Geom<D>;
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds[G::NSTAGE][G::TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds[G::NSTAGE][G::TILE_BYTES];

  const Rows r = rows_of(p);
  const AttnUnit& u = r.u;
  if (u.key_end <= u.key_begin) return;  // padding entry: uniform exit
  const int lane = r.lane, wave = r.wave, h = r.h, qpos = r.qpos;
  const Ctx c{(const_i32_ptr)p.page_ids + u.page_base, p.k_pool, p.v_pool, p.num_kv_heads, u.page_base, u.key_end,
              r.kv_head};
  const float scale = p.scale_log2;  // softmax scale of the scores in log2 units

  bf16x8 qf[G::KSTEPS];
  load_q<D, SQ>(qf, p, r, scale);
  int koff[G::KSTEPS];
  k_offsets<D>(koff, r.n, h);
  const int vbase = v_offset(r.n, h);
  LoadSlot<D> slot[G::PER_WAVE];
#pragma unroll
  for (int it = 0; it < G::PER_WAVE; it++) slot[it].init(it * kWaves + wave, lane);

  f32x16 o[G::DB];
  // running maximum (log2 units) and sum of the lane's row; folded: m relative to the
  // first tile's row maximum, and -m as the score tiles' accumulator input
  float m_run, l_run, mx;
  f32x16 c0;

  const int kb0 = u.key_begin;
  const int n_tiles = (u.key_end - kb0 + kBN - 1) / kBN;
  // tiles [0, n_full) hold keys every row of the unit sees; later ones need the causal mask
  int n_full = (u.q_pos0 + 1 - kb0) / kBN;
  n_full = n_full < 0 ? 0 : (n_full > n_tiles ? n_tiles : n_full);
  const int last_whole = (u.key_end - kb0) / kBN;  // tiles [0, last_whole) lie inside [kb0, key_end)

  // Issue this wave's pieces of K(tk) and V(tv) into the ring (tk / tv < 0: skip):
  // direct loads, except for a V tile reaching past key_end, which is loaded, zeroed
  // and written synchronously (V pieces go first, so that wait only covers older
  // loads).  Returns the direct loads issued.
  // Per slot: the pool base of this KV head, and the page id of the tile the slot
  // loads next (read one iteration ahead, so the scalar load is off the critical path).
  const uint32_t page_bytes = (uint32_t)p.num_kv_heads * (kPageSize * D * 2);
  const char* head_base[G::PER_WAVE];
  uint32_t pid[G::PER_WAVE];
#pragma unroll
  for (int it = 0; it < G::PER_WAVE; it++)
    head_base[it] = (const char*)(it >= G::K_SLOTS ? p.v_pool : p.k_pool) + (size_t)r.kv_head * (kPageSize * D * 2);
  const int lp0 = (int)((uint32_t)kb0 / kPageSize);
  auto page_for = [&](int it, int t) -> uint32_t {
    return (uint32_t)page_of(c, lp0 + t * (kBN / kPageSize) + slot[it].page_sel);
  };
  auto issue = [&](int tk, int tv) -> int {
    int direct = 0;
#pragma unroll
    for (int it = G::PER_WAVE - 1; it >= 0; it--) {
      const LoadSlot<D>& s = slot[it];
      const bool is_v = it >= G::K_SLOTS;
      const int t = is_v ? tv : tk;
      if (t < 0) continue;
      const char* block = page_block(head_base[it], pid[it], page_bytes);
      uint8_t* tile = is_v ? v_lds[t % G::NSTAGE] : k_lds[t % G::NSTAGE];
      if (is_v && t >= last_whole) {
        *(uint4*)(tile + s.j * 1024 + lane * 16) =
            mask_v_tail<D>(*(const uint4*)(block + s.off), s, kb0 + t * kBN, u.key_end);
      } else {
        issue_direct<D>(s, block, tile);
        direct++;
      }
      pid[it] = page_for(it, t + 1);  // next iteration's tile for this slot
    }
    return direct;
  };

  // One pass over the unit.  FIXED: the reference point stays at the first tile's
  // row maximum (no per-tile maximum, no rescale); otherwise it moves lazily.
  auto run = [&](auto fixed) {
    constexpr bool FIXED = decltype(fixed)::value;
#pragma unroll
    for (int b = 0; b < G::DB; b++) o[b] = f32x16{};
    m_run = SQ ? 0.0f : -1e30f;
    l_run = 0.0f;
    c0 = f32x16{};
    // ---- prologue: K(0), K(1), V(0) resident; K(2), V(1) and then K(3), V(2) in flight
    // (they play the loads of iterations -2 and -1)
    auto tile_or_none = [&](int t) { return t < n_tiles ? t : -1; };
    int issued_prev = 0;
#pragma unroll
    for (int it = 0; it < G::PER_WAVE; it++) pid[it] = page_for(it, 0);
    issue(0, 0);
#pragma unroll
    for (int it = 0; it < G::PER_WAVE; it++) pid[it] = page_for(it, 1);
    issue(tile_or_none(1), -1);
    wait_vmcnt<0>();
#pragma unroll
    for (int it = 0; it < G::PER_WAVE; it++) pid[it] = page_for(it, it >= G::K_SLOTS ? 1 : 2);
    issue(tile_or_none(2), tile_or_none(1));
    issued_prev = issue(tile_or_none(3), tile_or_none(2));  // pid already advanced to K(3), V(2)
    __syncthreads();

    f32x16 sa[kKB], sb[kKB];
    bf16x8 pb[2 * kKB];
    qk_tile<D>(sa, k_lds[0], koff, qf, c0);
    mx = n_full > 0 ? row_max<false>(sa, kb0, qpos, h) : row_max<true>(sa, kb0, qpos, h);
    if constexpr (SQ) set_reference(sa, mx, m_run, c0);
    else if constexpr (FIXED) m_run = mx * scale;
    if constexpr (FIXED && !SQ) prescale(sa, scale, m_run);
    __syncthreads();  // every wave has read K(0) before iteration 0 refills its slot with K(4)

    // lazy rescale before the scores of the tile whose maximum is mx are exponentiated:
    // the reference maximum moves only when a row outgrows it by 2^8
    auto rescale = [&](f32x16 (&st)[kKB]) {
      if constexpr (SQ) {
        folded_rescale<D>(st, o, mx, m_run, l_run, c0);
      } else if (__any(mx * scale > m_run + kRescaleThreshold)) {
        const float m_new = fmaxf(m_run, mx * scale);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int b = 0; b < G::DB; b++) o[b] *= alpha;
        m_run = m_new;
      }
    };

    // One pipelined iteration: consumes S(t) (scores in s_cur; in the second pass its
    // maximum in mx), produces S(t+1) into s_nxt (and its maximum), accumulates
    // P(t) V(t).  Issues K(t+4) and V(t+3) into the ring and, before its barrier,
    // waits for K(t+2) and V(t+1), which were issued two iterations earlier.
    // In the unmasked variant tile t+1 exists and needs no mask, so the compute part
    // is one branch-free block in which MFMA and the softmax VALU work interleave.
    auto iteration = [&](f32x16 (&s_cur)[kKB], f32x16 (&s_nxt)[kKB], int t, auto masked, auto whole, auto stage) {
      constexpr bool MASKED = decltype(masked)::value;
      constexpr bool WHOLE = decltype(whole)::value;
      constexpr int ST = decltype(stage)::value;
      // ring slot of tile t + d: a constant when the caller knows t's slot, so every
      // LDS operand address is a register plus an immediate offset
      auto ring = [&](int d) -> int {
        if constexpr (ST >= 0) return (ST + d) % G::NSTAGE;
        else return (t + d) % G::NSTAGE;
      };
      const int k0 = kb0 + t * kBN;
      const bool has_next = MASKED ? t + 1 < n_tiles : true;
      const int tk = WHOLE || t + 4 < n_tiles ? t + 4 : -1;
      const int tv = WHOLE || t + 3 < n_tiles ? t + 3 : -1;
      int issued = G::PER_WAVE;
      constexpr bool SPREAD = WHOLE && !MASKED;  // steady state
      const char* blk[G::PER_WAVE];
      if constexpr (SPREAD) {
#pragma unroll
        for (int it = 0; it < G::PER_WAVE; it++) blk[it] = page_block(head_base[it], pid[it], page_bytes);
      } else {
        issued = issue(tk, tv);
      }

      if constexpr (!FIXED) rescale(s_cur);
      // Exact form with the fixed reference: S(t) already holds s * scale - m, formed
      // one iteration earlier beside the PV products (which have no other VALU
      // work) by the same FMA exp_pack would use.
      constexpr bool PRE = FIXED && !SQ;

      if constexpr (MASKED) {
        if (has_next) qk_tile<D>(s_nxt, k_lds[ring(1)], koff, qf, c0);
        l_run = exp_pack<SQ || PRE>(s_cur, pb, l_run, m_run, scale);
        pv_tile<D>(o, v_lds[ring(0)], vbase, pb);
        if (has_next) {
          if constexpr (FIXED) causal_mask(s_nxt, k0 + kBN, qpos, h);
          else mx = row_max<true>(s_nxt, k0 + kBN, qpos, h);
          if constexpr (PRE) prescale(s_nxt, scale, m_run);
        }
      } else if constexpr (SPREAD) {
        qk_tile<D>(s_nxt, k_lds[ring(1)], koff, qf, c0, [&](int i) {
          const int it = G::PER_WAVE - 1 - i;
          const bool is_v = it >= G::K_SLOTS;
          issue_direct<D>(slot[it], blk[it], is_v ? v_lds[ring(3)] : k_lds[ring(4)]);  // V(t+3), K(t+4)
        });
        l_run = exp_pack<SQ || PRE>(s_cur, pb, l_run, m_run, scale);
        pv_tile<D>(o, v_lds[ring(0)], vbase, pb);
        if constexpr (!FIXED) mx = row_max<false>(s_nxt, k0 + kBN, qpos, h);
        if constexpr (PRE) prescale(s_nxt, scale, m_run);
      } else {
        qk_tile<D>(s_nxt, k_lds[ring(1)], koff, qf, c0);
        l_run = exp_pack<SQ || PRE>(s_cur, pb, l_run, m_run, scale);
        pv_tile<D>(o, v_lds[ring(0)], vbase, pb);
        if constexpr (!FIXED) mx = row_max<false>(s_nxt, k0 + kBN, qpos, h);
        if constexpr (PRE) prescale(s_nxt, scale, m_run);
      }

      if constexpr (SPREAD) {
        // next page ids, read after this iteration's last LDS operand read so that no
        // operand wait has to cover an outstanding scalar load
#pragma unroll
        for (int it = 0; it < G::PER_WAVE; it++) pid[it] = page_for(it, (it >= G::K_SLOTS ? tv : tk) + 1);
      }
      // K(t+2), V(t+1) (issued two iterations ago) must be in LDS before the barrier
      if constexpr (WHOLE) wait_vmcnt<2 * G::PER_WAVE>();
      else wait_issued<2 * G::PER_WAVE>(issued + issued_prev);
      issued_prev = issued;
      // Nothing crosses the barrier in the schedule (folded form, and the exact
      // form's fixed-reference pass).  Left free, the compiler moves a tile's
      // register-only exponentials into the next iteration, which then carries
      // twice the VALU work beside its products while the one before has none.
      if constexpr (SQ || FIXED) __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      if constexpr (SQ || FIXED) __builtin_amdgcn_sched_barrier(0);
    };

    int t = 0;
    // unmasked part: S(t+1) needs no mask while t + 1 < n_full.  While the tiles an
    // iteration issues (K(t+4), V(t+3)) are whole, the loads are unconditional; the
    // prologue issued K(3) and V(2) in full whenever that holds for t = 0.
    {
      const int whole_end = (last_whole - 3 < n_tiles - 4 ? last_whole - 3 : n_tiles - 4);
      // four tiles per trip (t % 4 == 0 at its top): every ring slot is a constant
      for (; t + 4 < n_full && t + 3 < whole_end; t += 4) {
        iteration(sa, sb, t, False{}, True{}, Stage<0>{});
        iteration(sb, sa, t + 1, False{}, True{}, Stage<1>{});
        iteration(sa, sb, t + 2, False{}, True{}, Stage<2>{});
        iteration(sb, sa, t + 3, False{}, True{}, Stage<3>{});
      }
      for (; t + 2 < n_full && t + 1 < whole_end; t += 2) {
        iteration(sa, sb, t, False{}, True{}, AnyStage{});
        iteration(sb, sa, t + 1, False{}, True{}, AnyStage{});
      }
    }
    for (; t + 2 < n_full; t += 2) {
      iteration(sa, sb, t, False{}, False{}, AnyStage{});
      iteration(sb, sa, t + 1, False{}, False{}, AnyStage{});
    }
    if (t + 1 < n_full) {
      iteration(sa, sb, t, False{}, False{}, AnyStage{});
      t++;
#pragma unroll
      for (int kb = 0; kb < kKB; kb++) sa[kb] = sb[kb];
    }
    for (; t < n_tiles; t += 2) {
      iteration(sa, sb, t, True{}, False{}, AnyStage{});
      if (t + 1 < n_tiles) iteration(sb, sa, t + 1, True{}, False{}, AnyStage{});
    }

    wait_vmcnt<0>();  // no load into this workgroup's LDS may outlive it
  };

  // Against a fixed reference the sums are exact unless a later score outgrew the
  // first tile's maximum far enough to overflow; then the whole workgroup runs the
  // unit again with the moving reference.
  run(True{});
  const bool bad = __any(r.valid && !all_finite<D>(o, l_run));
  __syncthreads();  // the ring is free
  int* vote = (int*)&k_lds[0][0];
  if (lane == 0) vote[wave] = bad ? 1 : 0;
  __syncthreads();
  int again = 0;
#pragma unroll
  for (int w = 0; w < kWaves; w++) again |= vote[w];
  if (again) {
    __syncthreads();  // every wave has read the votes before the ring refills
    run(False{});
  }
  write_result<D>(p, r, o, l_run, m_run, 1.0f);
}

// ---------------------------------------------------------------- fp8 pool
//
// The e4m3 codes of K(t) and V(t) come straight from the pool into a 4-slot LDS
// staging ring (global_load_lds_dwordx4, 1 KiB of codes per wave-wide load, half
// the loads of a bf16 tile), in the pool's own order: a K tile as 64 rows of D
// codes, a V tile as [page][dim][16 slots].  Staging slot s holds the "pair"
// s = {K(s+1), V(s)} (K runs one tile ahead, as in the products).  Every CU
// converts each code once: iteration t converts pair t+1 -- K(t+2) into bf16 K
// buffer t % 2 and V(t+1) into V^T buffer (t+1) % 2, in the layouts the bf16
// kernel uses -- while it multiplies K(t+1) and V(t) from the other buffers, so
// two bf16 buffers of each suffice.  Pair t+3 is loaded in iteration t, waited for
// at the end of iteration t+1 and, after that iteration's barrier, converted in
// iteration t+2 (each load has the rest of its iteration and the next one to land).
// The conversion is exact
// (every e4m3 value is a bf16 value); k_scale is folded into Q with the softmax
// scale, v_scale into the epilogue.

template <int D>
struct Geom8 {
  static constexpr int TILE_CODES = kBN * D;              // bytes of codes of one K (or V) tile
  static constexpr int PAIR = 2 * TILE_CODES;             // a staging slot: K codes, then V codes
  static constexpr int KINSTR = TILE_CODES / 1024;        // 1 KiB direct loads per tile
  static constexpr int NDMA = 2 * KINSTR / kWaves;        // direct loads per wave and pair
  static constexpr int CPR16 = D / 16;                    // 16-code chunks per K row
  static constexpr int NSTG = 4;                          // staging slots
  static constexpr int NBUF = 2;                          // bf16 buffers of K and of V^T
  static_assert(NDMA >= 1 && (2 * KINSTR) % kWaves == 0, "direct loads must spread evenly over waves");
};

// One wave's direct load of a pair: load g = wave + 8 * it is K load g (g < KINSTR)
// or V load g - KINSTR; lane l of load j moves 16 codes to staging byte
// 1024 j + 16 l of the tile's region.
template <int D>
struct CodeLoad {
  bool is_v;
  int j;
  int off;       // byte offset of the lane's 16 codes inside the (page, head) block
  int page_sel;  // page of the tile
  __device__ __forceinline__ void init(int g, int lane) {
    using G8 = Geom8<D>;
    is_v = g >= G8::KINSTR;
    j = is_v ? g - G8::KINSTR : g;
    const int q = 64 * j + lane;
    if (is_v) {  // [page][dim][16 slots]: chunk q = (page q / D, dim q % D)
      page_sel = q / D;
      off = (q % D) * kPageSize;
    } else {     // 64 rows of D codes: chunk q = (key q / CPR16, 16 dims q % CPR16)
      const int key = q / G8::CPR16;
      page_sel = key / kPageSize;
      off = (key % kPageSize) * D + (q % G8::CPR16) * 16;
    }
    // a load's 64 chunks lie in one page (D >= 64): the same for every lane, which
    // keeps the page-id lookups scalar
    page_sel = __builtin_amdgcn_readfirstlane(page_sel);
  }
};

// Conversion of a pair by lane L = wave * 64 + lane of the workgroup: for k < NCONV
// it writes bf16 chunk Q = L + 512 k (16 bytes at 16 Q) of the K tile and of the
// V^T tile, so that the 8 lanes of each group write one 128-byte half of a row
// (LDS writes free of bank conflicts), and reads the 8 codes that chunk holds from
// where the tile's swizzle puts them:
//   K: chunk p = Q % CPR of row r = Q / CPR holds dims 8 c .. 8 c + 7, c = p ^ (r % CPR):
//      codes at byte r D + 8 c of the K codes;
//   V^T: half h = Q & 1 of dim row d = Q / 2 (page d / D) holds slots 8 s .. 8 s + 7,
//      s = h ^ ((d >> 3) & 1): codes at byte 16 d + 8 s of the V codes.
// Chunk Q + 512 sits 4096 code bytes further in both (the row swizzle repeats), and
// its V slots 4096 / D keys later.
template <int D>
struct ConvLane {
  static constexpr int NCONV = Geom<D>::TILE_BYTES / 16 / kAttnThreads;  // chunks per lane and tile
  static_assert(NCONV >= 1 && Geom<D>::TILE_BYTES % (16 * kAttnThreads) == 0, "conversion must spread evenly");
  static_assert(NCONV == 1 || (kAttnThreads / Geom<D>::CPR) % Geom<D>::CPR == 0, "swizzle repeats every 512 chunks");
  int ksrc;  // byte offset of the lane's K codes in the K codes of a staging slot
  int vsrc;  // byte offset of the lane's V codes in the V codes
  int vkey;  // key offset of the lane's first V slot in the tile
  __device__ __forceinline__ void init(int L) {
    using G = Geom<D>;
    const int r = L / G::CPR, pch = L % G::CPR;
    ksrc = r * D + ((pch ^ (r % G::CPR)) * 8);
    const int d = L / 2, hs = (L & 1) ^ ((d >> 3) & 1);
    vsrc = d * 16 + 8 * hs;
    vkey = (d / D) * kPageSize + 8 * hs;
  }
};

// Zero the bf16 values of V^T slots at or past key_end (8 slots starting at key).
__device__ __forceinline__ uint4 zero_past(uint4 x, int key, int key_end) {
  uint32_t* xw = (uint32_t*)&x;
#pragma unroll
  for (int e = 0; e < 4; e++) {
    const uint32_t lo = (key + 2 * e < key_end) ? 0xFFFFu : 0u;
    const uint32_t hi = (key + 2 * e + 1 < key_end) ? 0xFFFF0000u : 0u;
    xw[e] &= (lo | hi);
  }
  return x;
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 1) void extend_attn_fp8_kernel(AttnParams p) {
  using G = Geom<D>;
  using G8 = Geom8<D>;
  // one block, bf16 buffers first: every MFMA operand read and conversion write then
  // lies below 64 KiB and addresses with an immediate offset
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * G8::NBUF * G::TILE_BYTES + G8::NSTG * G8::PAIR];
  uint8_t(*k_lds)[G::TILE_BYTES] = (uint8_t(*)[G::TILE_BYTES])lds;
  uint8_t(*v_lds)[G::TILE_BYTES] = (uint8_t(*)[G::TILE_BYTES])(lds + G8::NBUF * G::TILE_BYTES);
  uint8_t(*stg)[G8::PAIR] = (uint8_t(*)[G8::PAIR])(lds + 2 * G8::NBUF * G::TILE_BYTES);

  const Rows r = rows_of(p);
  const AttnUnit& u = r.u;
  if (u.key_end <= u.key_begin) return;  // padding entry: uniform exit
  const int lane = r.lane, wave = r.wave, h = r.h, qpos = r.qpos;
  const Ctx c{(const_i32_ptr)p.page_ids + u.page_base, p.k_pool, p.v_pool, p.num_kv_heads, u.page_base, u.key_end,
              r.kv_head};
  // Q times softmax scale (log2 units) times k_scale: the products come out in the
  // exponent's units
  const float vscale = p.v_scale[r.kv_head];
  bf16x8 qf[G::KSTEPS];
  load_q<D, true>(qf, p, r, p.scale_log2 * p.k_scale[r.kv_head]);
  int koff[G::KSTEPS];
  k_offsets<D>(koff, r.n, h);
  const int vbase = v_offset(r.n, h);

  f32x16 o[G::DB];
  // running maximum m of the lane's row (log2 units), -m as the score tiles'
  // accumulator input; m starts at the first tile's row maximum
  float m_run, l_run, mx;
  f32x16 cneg;

  const int kb0 = u.key_begin;
  const int n_tiles = (u.key_end - kb0 + kBN - 1) / kBN;
  int n_full = (u.q_pos0 + 1 - kb0) / kBN;
  n_full = n_full < 0 ? 0 : (n_full > n_tiles ? n_tiles : n_full);
  const int last_whole = (u.key_end - kb0) / kBN;

  // direct loads: per wave, the pool base of this KV head and the page id of the
  // tile each load fetches next (read one pair ahead)
  const uint32_t page_bytes = (uint32_t)p.num_kv_heads * (kPageSize * D);
  CodeLoad<D> ld[G8::NDMA];
  const char* head_base[G8::NDMA];
  uint32_t pid[G8::NDMA];
#pragma unroll
  for (int it = 0; it < G8::NDMA; it++) {
    ld[it].init(wave + kWaves * it, lane);
    head_base[it] = (const char*)(ld[it].is_v ? p.v_pool : p.k_pool) + (size_t)r.kv_head * (kPageSize * D);
  }
  // the bf16 chunks this lane converts: 16 L (+ 8192 k) of each tile
  const int L = wave * 64 + lane;
  ConvLane<D> cv;
  cv.init(L);
  const int lp0 = (int)((uint32_t)kb0 / kPageSize);
  // tile of pair s that load `it` fetches: K(s+1) or V(s)
  auto tile_of = [&](int it, int s) { return ld[it].is_v ? s : s + 1; };
  auto page_for = [&](int it, int tt) -> uint32_t {  // tt >= 0
    return (uint32_t)page_of(c, lp0 + tt * (kBN / kPageSize) + ld[it].page_sel);
  };
  auto dma = [&](int it, uint8_t* slot, const char* block) {
    const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)(
        slot + (ld[it].is_v ? G8::TILE_CODES : 0) + ld[it].j * 1024);
    lds_dma_16(block, ld[it].off, lds);
  };
  // load pair s (tiles that do not exist are skipped); returns the loads issued
  auto issue = [&](int s) -> int {
    int n = 0;
#pragma unroll
    for (int it = 0; it < G8::NDMA; it++) {
      const int tt = tile_of(it, s);
      if (tt < 0 || tt >= n_tiles) continue;
      dma(it, stg[s & 3], page_block(head_base[it], pid[it], page_bytes));
      n++;
      pid[it] = page_for(it, tt + 1);
    }
    return n;
  };
  // convert pair s from staging slot `src` into the bf16 buffers kdst (K(s+1)) and
  // vdst (V(s))
  auto convert = [&](int s, auto whole, const uint8_t* src, uint8_t* kdst, uint8_t* vdst) {
    constexpr bool WHOLE = decltype(whole)::value;
    const bool k_in = WHOLE || (s + 1 >= 0 && s + 1 < n_tiles);  // K(s+1) exists
    const bool v_in = WHOLE || (s >= 0 && s < n_tiles);          // V(s) exists
#pragma unroll
    for (int k = 0; k < ConvLane<D>::NCONV; k++) {
      if (k_in) {
        const uint2 c = *(const uint2*)(src + cv.ksrc + 4096 * k);
        *(uint4*)(kdst + 16 * L + 8192 * k) = fp8x8_to_bf16x8(c);
      }
      if (v_in) {
        const uint2 c = *(const uint2*)(src + G8::TILE_CODES + cv.vsrc + 4096 * k);
        uint4 x = fp8x8_to_bf16x8(c);
        if (!WHOLE && s >= last_whole) x = zero_past(x, kb0 + s * kBN + cv.vkey + (4096 / D) * k, u.key_end);
        *(uint4*)(vdst + 16 * L + 8192 * k) = x;
      }
    }
  };

  // One pass over the unit.  FIXED: the reference point stays at the first tile's
  // row maximum (no per-tile maximum, no rescale); otherwise it moves lazily.
  auto run = [&](auto fixed) {
    constexpr bool FIXED = decltype(fixed)::value;
#pragma unroll
    for (int b = 0; b < G::DB; b++) o[b] = f32x16{};
    m_run = 0.0f;
    l_run = 0.0f;
    cneg = f32x16{};
    // ---- prologue: pairs -1 = {K(0)}, 0, 1, 2 loaded; -1 and 0 converted (K(0), K(1),
    // V(0) in bf16), 1 resident, 2 in flight
#pragma unroll
    for (int it = 0; it < G8::NDMA; it++) pid[it] = page_for(it, 0);
    issue(-1);
    issue(0);
    issue(1);
    const int in_flight = issue(2);
    wait_issued<G8::NDMA>(in_flight);
    __syncthreads();
    convert(-1, False{}, stg[3], k_lds[0], v_lds[1]);
    convert(0, False{}, stg[0], k_lds[1], v_lds[0]);
    __syncthreads();

    f32x16 sa[kKB], sb[kKB];
    bf16x8 pb[2 * kKB];
    qk_tile<D>(sa, k_lds[0], koff, qf, cneg);
    mx = n_full > 0 ? row_max<false>(sa, kb0, qpos, h) : row_max<true>(sa, kb0, qpos, h);
    set_reference(sa, mx, m_run, cneg);
    __syncthreads();  // every wave has read K(0) before iteration 0 converts K(2) into its buffer


    // One pipelined iteration: consumes S(t), produces S(t+1) from bf16 K(t+1) (in the
    // second pass with its maximum), accumulates P(t) V(t), loads pair t+3 and
    // converts pair t+1.  Before the barrier only this iteration's loads may still be
    // in flight.
    auto iteration = [&](f32x16 (&s_cur)[kKB], f32x16 (&s_nxt)[kKB], int t, auto masked, auto whole, auto stage) {
      constexpr bool MASKED = decltype(masked)::value;
      constexpr bool WHOLE = decltype(whole)::value;
      constexpr int ST = decltype(stage)::value;
      auto buf = [&](int d) -> int {  // bf16 buffer of tile t + d
        if constexpr (ST >= 0) return (ST + d) % G8::NBUF;
        else return (t + d) % G8::NBUF;
      };
      auto slot_of = [&](int d) -> int {  // staging slot of pair t + d
        if constexpr (ST >= 0) return (ST + d) % G8::NSTG;
        else return (t + d) % G8::NSTG;
      };
      const int k0 = kb0 + t * kBN;
      const bool has_next = MASKED ? t + 1 < n_tiles : true;
      constexpr bool SPREAD = WHOLE && !MASKED;
      int issued = G8::NDMA;
      const char* blk[G8::NDMA];
      if constexpr (SPREAD) {
#pragma unroll
        for (int it = 0; it < G8::NDMA; it++) blk[it] = page_block(head_base[it], pid[it], page_bytes);
      } else {
        issued = issue(t + 3);
      }
      if constexpr (!FIXED) folded_rescale<D>(s_cur, o, mx, m_run, l_run, cneg);
      if constexpr (SPREAD) {
        qk_tile<D>(s_nxt, k_lds[buf(1)], koff, qf, cneg, [&](int i) {
          if (i < G8::NDMA) dma(i, stg[slot_of(3)], blk[i]);
        });
      } else {
        if (!MASKED || has_next) qk_tile<D>(s_nxt, k_lds[buf(1)], koff, qf, cneg);
      }
      convert(t + 1, whole, stg[slot_of(1)], k_lds[buf(2)], v_lds[buf(1)]);
      l_run = exp_pack<true>(s_cur, pb, l_run, m_run, 0.0f);
      pv_tile<D>(o, v_lds[buf(0)], vbase, pb);
      if constexpr (MASKED) {
        if (has_next) {
          if constexpr (FIXED) causal_mask(s_nxt, k0 + kBN, qpos, h);
          else mx = row_max<true>(s_nxt, k0 + kBN, qpos, h);
        }
      } else if constexpr (!FIXED) {
        mx = row_max<false>(s_nxt, k0 + kBN, qpos, h);
      }
      if constexpr (SPREAD) {
#pragma unroll
        for (int it = 0; it < G8::NDMA; it++) pid[it] = page_for(it, tile_of(it, t + 4));
      }
      // pair t+2 (loaded one iteration ago) is converted in the next iteration
      if constexpr (WHOLE) wait_vmcnt<G8::NDMA>();
      else wait_issued<G8::NDMA>(issued);
      // each iteration keeps its own softmax work (as in the bf16 kernel's folded form)
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
    };

    int t = 0;
    {
      // steady state: the pair loaded (t+3: K(t+4), V(t+3)) exists and the pair
      // converted (t+1: K(t+2), V(t+1)) needs no zeroing
      const int whole_end = (n_tiles - 4 < last_whole - 1 ? n_tiles - 4 : last_whole - 1);
      for (; t + 4 < n_full && t + 3 < whole_end; t += 4) {
        iteration(sa, sb, t, False{}, True{}, Stage<0>{});
        iteration(sb, sa, t + 1, False{}, True{}, Stage<1>{});
        iteration(sa, sb, t + 2, False{}, True{}, Stage<2>{});
        iteration(sb, sa, t + 3, False{}, True{}, Stage<3>{});
      }
      for (; t + 2 < n_full && t + 1 < whole_end; t += 2) {
        iteration(sa, sb, t, False{}, True{}, AnyStage{});
        iteration(sb, sa, t + 1, False{}, True{}, AnyStage{});
      }
    }
    for (; t + 2 < n_full; t += 2) {
      iteration(sa, sb, t, False{}, False{}, AnyStage{});
      iteration(sb, sa, t + 1, False{}, False{}, AnyStage{});
    }
    if (t + 1 < n_full) {
      iteration(sa, sb, t, False{}, False{}, AnyStage{});
      t++;
#pragma unroll
      for (int kb = 0; kb < kKB; kb++) sa[kb] = sb[kb];
    }
    for (; t < n_tiles; t += 2) {
      iteration(sa, sb, t, True{}, False{}, AnyStage{});
      if (t + 1 < n_tiles) iteration(sb, sa, t + 1, True{}, False{}, AnyStage{});
    }

    wait_vmcnt<0>();  // no load into this workgroup's LDS may outlive it
  };

  // as in the bf16 kernel: a fixed reference, and a second pass with the moving one
  // if anything overflowed
  run(True{});
  const bool bad = __any(r.valid && !all_finite<D>(o, l_run));
  __syncthreads();  // the staging ring and the bf16 buffers are free
  int* vote = (int*)&stg[0][0];
  if (lane == 0) vote[wave] = bad ? 1 : 0;
  __syncthreads();
  int again = 0;
#pragma unroll
  for (int w = 0; w < kWaves; w++) again |= vote[w];
  if (again) {
    __syncthreads();  // every wave has read the votes before the ring refills
    run(False{});
  }
  write_result<D>(p, r, o, l_run, m_run, vscale);
}

// Combine the parts of split tiles: o = sum_p e^{lse_p - M} o_p / sum_p e^{lse_p - M}.
// Rows of a tile per merge workgroup (256 lanes, one 16-byte column group each).
template <int D>
constexpr int kMergeRows = 256 / (D / 4);
static_assert(kTileRows % kMergeRows<128> == 0 && kTileRows % kMergeRows<64> == 0, "whole row blocks");

template <int D>
__global__ __launch_bounds__(256) void merge_kernel(MergeParams p) {
  // workgroup (merge, row block): kMergeRows rows of the tile, one 16-byte column
  // group of one row per lane, so that a merge of few tiles still spreads over the CUs
  const MergeUnit mu = p.merges[blockIdx.x];
  const int kv_head = mu.head_ntok >> 16;
  const int ntok = mu.head_ntok & 0xFFFF;
  constexpr int C4 = D / 4;
  const int rho = (int)blockIdx.y * kMergeRows<D> + (int)threadIdx.x / C4;
  const int c = ((int)threadIdx.x % C4) * 4;
  const int tok = rho / p.group;
  if (tok >= ntok) return;
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

}  // namespace

hipError_t launch_extend_attention(const AttnParams& p, int64_t n_units, int head_dim, bool fp8, bool scaled_q,
                                   hipStream_t stream) {
  if (n_units <= 0) return hipSuccess;
  dim3 grid((unsigned)n_units), block(kAttnThreads);
  if (head_dim == 128) {
    if (fp8) hipLaunchKernelGGL((extend_attn_fp8_kernel<128>), grid, block, 0, stream, p);
    else if (scaled_q) hipLaunchKernelGGL((extend_attn_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((extend_attn_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (fp8) hipLaunchKernelGGL((extend_attn_fp8_kernel<64>), grid, block, 0, stream, p);
    else if (scaled_q) hipLaunchKernelGGL((extend_attn_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((extend_attn_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_merge(const MergeParams& p, int64_t n_merges, int head_dim, hipStream_t stream) {
  if (n_merges <= 0) return hipSuccess;
  const dim3 block(256);
  if (head_dim == 128)
    hipLaunchKernelGGL((merge_kernel<128>), dim3((unsigned)n_merges, kTileRows / kMergeRows<128>), block, 0, stream, p);
  else
    hipLaunchKernelGGL((merge_kernel<64>), dim3((unsigned)n_merges, kTileRows / kMergeRows<64>), block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace kvx
