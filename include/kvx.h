/*
 * kvx.h -- prefix-extend attention over a paged KV pool on AMD MI355X (gfx950).
 *
 * The operation.  An agent that returns for another turn reuses the KV tensors
 * its cached prefix still holds and computes only the uncached suffix (paper,
 * Section 1 and Section 2, "Prefix caching for multi-turn agents"): prefill
 * materialises the suffix's K/V in the attention layer, and every suffix query
 * attends causally over the cached prefix and the suffix before it.  The number
 * of uncached tokens of a request is its prompt length minus its cached prefix
 * length (Section 4, metrics).  The host keeps the prefix index and the eviction
 * policy (Section 3.2, Algorithm 1); what reaches this library is, per request,
 * a prefix length P, an extend length E and a page table.
 *
 * Conventions shared by every call
 *   - Return value: KVX_OK (0) or a kvx_status code; kvx_last_error() then
 *     describes the failure (thread-local string).  No exception crosses the ABI.
 *   - Argument checks run synchronously on the host before anything is queued;
 *     a call that fails them queues no work and leaves all buffers untouched.
 *   - Device work is queued on `stream` (a hipStream_t; NULL = the null stream)
 *     and is asynchronous: caller-owned buffers must stay alive until the
 *     stream reaches the call.  Calls on one stream execute in order.
 *   - A pool owns one plan buffer and one partial-result buffer, reused by
 *     every call on it.  Work on one pool must therefore be ordered: issue its
 *     calls on one stream, or make a second stream wait (hipStreamWaitEvent)
 *     for the first one's calls before queuing more on the pool.  Calls on one
 *     pool that overlap on two streams race on those buffers, and calls on one
 *     pool must come from one host thread at a time.  Separate pools are
 *     independent.
 *   - Calls build their work plan on the host and upload it through a pinned
 *     staging buffer, waiting on the host for that buffer's previous copy, and
 *     may allocate device scratch the first time a size is seen: they are not
 *     meant to be captured into a HIP graph.  Scratch grows with the
 *     stream-ordered allocator (hipMallocAsync / hipFreeAsync): growing never
 *     waits for the device on the host.
 *   - "host" pointers are ordinary CPU memory read during the call;
 *     "device" pointers are GPU memory (hipMalloc / torch CUDA tensors).
 *   - bf16 means IEEE binary32 truncated to its upper 16 bits (2 bytes).
 *   - Row buffers (Q, O, K_ext, V_ext, page I/O buffers, norm weights, spill
 *     records) must start 16-byte aligned (the kernels move 16-byte pieces);
 *     the argument checks reject other addresses with KVX_EINVAL.
 *   - Rows of Q, O, K_ext and V_ext are the suffix tokens of all requests,
 *     request by request: request r owns rows [sum_{s<r} E_s, sum_{s<=r} E_s).
 *   - Page ids outside [0, num_pages) are undefined behaviour unless the
 *     environment variable KVX_VALIDATE=1 is set, in which case the page table
 *     is copied to the host and checked (KVX_ERANGE), at the cost of a sync.
 */
#ifndef KVX_H
#define KVX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Query rows of one extend_attention work item: suffix tokens x the query heads
 * that share one KV head (tokens per item = KVX_TILE_ROWS / (Hq / Hkv)). */
#define KVX_TILE_ROWS 256

typedef struct kvx_pool kvx_pool; /* opaque; owned by the library */
typedef void *kvx_stream_t;       /* a hipStream_t */

enum kvx_status {
    KVX_OK = 0,
    KVX_EINVAL = 1,       /* bad argument (shape, length, null pointer, ...) */
    KVX_ENOMEM = 2,       /* device or host allocation failed */
    KVX_ERANGE = 3,       /* page id outside the pool (KVX_VALIDATE=1 only) */
    KVX_EUNSUPPORTED = 4, /* valid but unsupported configuration */
    KVX_EHIP = 5          /* a HIP runtime call failed */
};

enum kvx_kv_dtype {
    KVX_KV_BF16 = 0,     /* K/V stored as bf16 */
    KVX_KV_FP8_E4M3 = 1  /* K/V stored as OCP e4m3 (fp8, max 448, no inf) with per-head scales */
};

/* ------------------------------------------------------------------ the pool */

/* Device layout of a pool, for tests and tools.  Element strides.  K is stored
 * [page][kv_head][slot][dim]; V is stored transposed within a page,
 * [page][kv_head][dim][slot], so that one page of one head is a contiguous
 * block in both (4 KiB for bf16, head_dim 128). */
typedef struct {
    void *k_base;          /* device */
    void *v_base;          /* device */
    int64_t num_pages;
    int32_t page_size;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t kv_dtype;      /* enum kvx_kv_dtype */
    int32_t elem_bytes;    /* 2 (bf16) or 1 (fp8) */
    int32_t reserved;
    int64_t k_stride_page, k_stride_head, k_stride_slot, k_stride_dim;
    int64_t v_stride_page, v_stride_head, v_stride_slot, v_stride_dim;
    const float *k_scale;  /* device [num_kv_heads], NULL for bf16 */
    const float *v_scale;  /* device [num_kv_heads], NULL for bf16 */
} kvx_pool_layout;

/*
 * Allocate a KV pool of `num_pages` pages of `page_size` tokens: the one pool of
 * fixed-size pages from which every request's reusable KV is served (Section 2,
 * on how serving systems keep cached KV).
 *   page_size     must be 16.
 *   num_kv_heads  >= 1.
 *   head_dim      64 or 128.
 *   kv_dtype      KVX_KV_BF16 or KVX_KV_FP8_E4M3.
 *   k_scale, v_scale  host [num_kv_heads] positive finite dequantisation scales
 *                 for the fp8 pool (stored value = code * scale); NULL for bf16.
 *   out           receives the handle.
 * The pool's contents are zero after creation.  Synchronous.  Errors: EINVAL,
 * EUNSUPPORTED (page_size != 16, head_dim not 64/128), ENOMEM, EHIP.
 */
int kv_pool_create(int64_t num_pages, int32_t page_size, int32_t num_kv_heads, int32_t head_dim,
                   int32_t kv_dtype, const float *k_scale, const float *v_scale, kvx_pool **out);

/* Free a pool (waits for the device to go idle first).  NULL is a no-op. */
int kv_pool_destroy(kvx_pool *pool);

/* Fill *out with the pool's device layout.  Errors: EINVAL. */
int kv_pool_layout(const kvx_pool *pool, kvx_pool_layout *out);

/*
 * Raw page upload / readback in the canonical order [n][kv_head][slot][dim]
 * for both K and V, in the pool's element type (bf16 bits or fp8 codes); the
 * library converts to and from its own V layout.  Neither call converts values.
 *   page_ids   host [n] physical page ids (each in [0, num_pages); always checked)
 *   k_*, v_*   device buffers of n * num_kv_heads * page_size * head_dim elements
 * Asynchronous on `stream`.  Errors: EINVAL, ERANGE, ENOMEM, EHIP.
 */
int kv_pool_write_pages(kvx_pool *pool, const int32_t *page_ids, int64_t n, const void *k_src,
                        const void *v_src, kvx_stream_t stream);
int kv_pool_read_pages(const kvx_pool *pool, const int32_t *page_ids, int64_t n, void *k_dst,
                       void *v_dst, kvx_stream_t stream);

/*
 * KV spill to host memory and reload, instead of recomputing an evicted tail
 * (the paper's stated future work, Section 6: keep evicted KV in a slower tier
 * and bring it back).  A spill record holds one page exactly as the pool holds
 * it -- its K block then its V block, kv_pool_record_bytes() bytes, raw (bf16 or
 * fp8 codes; the scales stay with the pool) -- so spill + reload is a bit-exact
 * round trip into any page of a pool of the same shape and dtype.
 *   kv_pool_spill:  record slots[i] of host := page page_ids[i]
 *   kv_pool_reload: page page_ids[i] := record slots[i] of host
 * page_ids, slots: host [n]; page ids in [0, num_pages), slots in [0, host_slots);
 *   the written side may not repeat (slots of a spill, page ids of a reload).
 * host: pinned host memory (hipHostMalloc or a pinned torch tensor) of at least
 *   host_slots records; the kernel reaches it over the host link.  Asynchronous
 *   on `stream`: the host buffer and pool pages must not be touched until the
 *   stream has passed the call.  Errors: EINVAL (also unpinned host memory),
 *   ERANGE, ENOMEM, EHIP.  n = 0: no-op.
 */
int kv_pool_record_bytes(const kvx_pool *pool, int64_t *bytes);
int kv_pool_spill(const kvx_pool *pool, const int32_t *page_ids, const int32_t *slots, int64_t n,
                  void *host, int64_t host_slots, kvx_stream_t stream);
int kv_pool_reload(kvx_pool *pool, const int32_t *page_ids, const int32_t *slots, int64_t n,
                   const void *host, int64_t host_slots, kvx_stream_t stream);

/* ---------------------------------------------------------------- the batch */

/* One prefix-extend batch.  Request r has a cached prefix of P_r tokens already
 * in the pool and an uncached suffix of E_r tokens; its logical pages
 * j = 0 .. ceil((P_r+E_r)/16)-1 are page_ids[page_indptr[r] + j]. */
typedef struct {
    int32_t num_reqs;              /* R >= 0 */
    const int32_t *prefix_lens;    /* host [R], P_r >= 0 */
    const int32_t *extend_lens;    /* host [R], E_r >= 0 */
    const int32_t *page_indptr;    /* host [R+1], non-decreasing, starts at 0; request r needs
                                      page_indptr[r+1]-page_indptr[r] >= ceil((P_r+E_r)/16) */
    const int32_t *page_ids;       /* device [page_indptr[R]] physical page ids */
} kvx_batch;

/*
 * Write the suffix's K and V into the pool (prefill materialises KV in every
 * attention layer, Section 2): for each request r, suffix token i and KV head h,
 * the token at absolute position t = P_r + i goes to slot t % 16 of logical page
 * t / 16.  bf16 pool: the bits are copied.  fp8 pool: each element is stored as
 * e4m3(clamp(float(x) * float(1/scale_h), -448, 448)), rounded to nearest even.
 * Slots not written by the batch keep their contents.
 *   k_ext, v_ext  device bf16 [T, num_kv_heads, head_dim], T = sum E_r.
 * Must precede extend_attention of the same batch on the same stream.
 * Errors: EINVAL, ERANGE (validation mode), ENOMEM, EHIP.  R = 0 or T = 0: no-op.
 */
int store_kv(kvx_pool *pool, const kvx_batch *batch, const void *k_ext, const void *v_ext,
             kvx_stream_t stream);

/* Layout of the rotation planes of a head (see store_kv_rope). */
enum {
    KVX_ROPE_HALF = 0,        /* plane j = dims (j, j + rotary_dim/2): GPT-NeoX, Llama, Qwen */
    KVX_ROPE_INTERLEAVED = 1  /* plane j = dims (2j, 2j + 1): GPT-J */
};

typedef struct {
    double theta;            /* frequency base > 0: plane j turns theta^(-2j/rotary_dim) rad per position */
    const double *inv_freq;  /* host [rotary_dim/2] rates (rad per position, finite, >= 0) used instead of
                                theta -- scaled or extended frequency tables -- or NULL; read during the call */
    int32_t rotary_dim;      /* rotated leading dims of a head: a multiple of 16 in [16, head_dim];
                                the dims past it pass through */
    int32_t style;           /* KVX_ROPE_HALF or KVX_ROPE_INTERLEAVED */
    const void *q_norm;      /* device bf16 [head_dim] RMS-norm weight for every Q head, or NULL: no norm */
    const void *k_norm;      /* the same for every K head */
    float norm_eps;          /* finite, >= 0; added to the mean square */
} kvx_rope;

/*
 * store_kv with the steps that produce attention's queries and keys fused in.
 * The paper describes neither step; the models it serves (Section 4) normalise
 * and rotate Q and K before K is cached.  For suffix token i of request r, at
 * absolute position t = P_r + i, every Q head and K head row x is
 *   normalised, when a weight w is given:  y = x * w / sqrt(mean(x^2) + norm_eps)
 *   (mean over all head_dim dims), then rotated: each plane (a, b) of the first
 *   rotary_dim dims turns by t * f_j:  (a cos - b sin, a sin + b cos).
 * The rotated K is stored as store_kv stores K (bf16 round-to-nearest-even, or
 * e4m3 of float(y) * float(1/scale) on an fp8 pool); V is stored exactly as by
 * store_kv; the rotated Q goes to q_out as bf16 (round to nearest even).
 * Arithmetic is float32, with every angle reduced to one turn in float64 first,
 * and each result is rounded once.
 *   q, q_out     device bf16 [T, num_q_heads, head_dim]; q_out may be q itself
 *                (in place) but may not overlap it otherwise; both unused (may be
 *                NULL) when num_q_heads = 0, which rotates and stores K only
 *   k_ext, v_ext device bf16 [T, num_kv_heads, head_dim], T = sum E_r (not modified)
 * Must precede extend_attention of the same batch (which then takes q_out) on the
 * same stream.  Errors: EINVAL, ERANGE (validation mode), ENOMEM, EHIP.
 * R = 0 or T = 0: no-op after the argument checks.
 */
int store_kv_rope(kvx_pool *pool, const kvx_batch *batch, const kvx_rope *rope, const void *q,
                  int32_t num_q_heads, void *q_out, const void *k_ext, const void *v_ext,
                  kvx_stream_t stream);

/*
 * Prefix-extend attention: for each request r, suffix row i and query head hq,
 *   o = softmax_j(sm_scale * q . k_j) v_j  over keys j = 0 .. P_r + i
 * of the request's logical sequence in the pool (cached prefix, then the suffix
 * written by store_kv).  Query head hq reads KV head hq / (num_q_heads / num_kv_heads).
 * The result equals attention over the whole context; only the suffix is computed
 * (Section 1: reuse the cached prefix, compute the uncached suffix).
 *   q            device bf16 [T, num_q_heads, head_dim]
 *   num_q_heads  a multiple of the pool's num_kv_heads, with at most
 *                KVX_TILE_ROWS query heads per KV head
 *   sm_scale     softmax scale, finite and > 0 (usually 1/sqrt(head_dim))
 *   out          device bf16 [T, num_q_heads, head_dim] (round to nearest even)
 *   lse          device fp32 [T, num_q_heads] natural-log sum of exp of the scaled
 *                scores, or NULL
 * A decode step -- every request has at most one suffix token, and at most 16
 * query heads share a KV head -- runs a dedicated decode kernel (key chunks of
 * each request and KV head streamed from HBM); the result is the same operation.
 * Uses a library-owned device workspace (grown with hipMallocAsync when a batch
 * needs more than any earlier one; at most 2 GiB of partial results).  Errors: EINVAL, EUNSUPPORTED, ERANGE (validation
 * mode), ENOMEM, EHIP.  R = 0 or T = 0: no-op.
 */
int extend_attention(kvx_pool *pool, const kvx_batch *batch, const void *q, int32_t num_q_heads,
                     float sm_scale, void *out, float *lse, kvx_stream_t stream);

/*
 * extend_attention for callers that cannot allocate device memory during the
 * call: tight serving loops and harnesses that forbid hipMalloc.  It is still
 * not capturable into a HIP graph: each call builds its plan on the host and
 * copies it from a host vector that is freed when the call returns, so a
 * captured copy would read freed memory on replay.  Same arguments, operation, kernels and result as extend_attention
 * (bit for bit when both split the key ranges alike), but the work plan and the
 * partial results of split key ranges go into one fixed device array of the
 * library instead of the pool's staging buffer and workspace; the call makes no
 * device or pinned allocation (only host containers for the plan).  The plan is
 * copied from pageable host memory (hipMemcpyAsync, staged before the call
 * returns).
 *   The array holds KVX_NOALLOC_PLAN_BYTES of plan (32 B per work item) and
 *   KVX_NOALLOC_PARTS_BYTES of partial results; the planner splits key ranges
 *   only into as many parts as fit.  A batch whose plan does not fit is refused
 *   with EUNSUPPORTED on the host, before any device work.
 *   Each GPU the library runs on holds its own copy of the array (64 MiB) from
 *   the first call on it until the process ends.  Every call on one GPU shares
 *   that copy, and each call leaves its plan and partial results in it: calls
 *   that may overlap on one GPU (two streams, or two host threads) race and must
 *   be ordered by the caller, even on different pools.
 * Errors: EINVAL, EUNSUPPORTED, ERANGE (validation mode), EHIP.
 */
#define KVX_NOALLOC_PLAN_BYTES (8u << 20)
#define KVX_NOALLOC_PARTS_BYTES (56u << 20)
int extend_attention_noalloc(kvx_pool *pool, const kvx_batch *batch, const void *q, int32_t num_q_heads,
                             float sm_scale, void *out, float *lse, kvx_stream_t stream);

/* ---------------------------------------------------------- planning, tuning */

/* One work item of extend_attention: a tile of suffix tokens of one request and
 * one KV head (all of that head's query heads), over the key range [key_begin,
 * key_end) of the request's logical sequence.  part >= 0 marks one part of a
 * key range split across workgroups (merged afterwards by log-sum-exp). */
typedef struct {
    int32_t req;
    int32_t kv_head;
    int32_t tok_begin;   /* first suffix token of the tile */
    int32_t tok_count;   /* suffix tokens in the tile */
    int32_t key_begin;
    int32_t key_end;
    int32_t part;        /* -1: whole range; else index of the partial result */
    int32_t xcd;         /* the XCD (L2 domain) the item is dispatched to */
} kvx_work_item;

/*
 * The host-side work plan extend_attention would launch for a batch (host only,
 * no device work): ragged (P, E) pairs cut into tiles, long key ranges split,
 * items ordered longest first within each XCD; for a decode step, key chunks of
 * every (request, KV head), longest first (tok_count 1).  Writes at most `cap` items to
 * `items` (may be NULL) and the total count to *count.
 *   num_kv_heads, num_q_heads, head_dim as for extend_attention.
 *   split_keys   as set by kv_pool_set_split_keys (0 = automatic).
 * Errors: EINVAL, EUNSUPPORTED.
 */
int extend_attention_plan(const kvx_batch *batch, int32_t num_q_heads, int32_t num_kv_heads,
                          int32_t head_dim, int32_t split_keys, kvx_work_item *items, int64_t cap,
                          int64_t *count);

/*
 * Key-range split length of extend_attention on this pool (tokens, a multiple
 * of 64, or 0 = automatic, the default).  A non-zero value splits every key
 * range longer than it (a decode step: chunks of that many keys); used to
 * exercise the split path.  A setting of the pool: takes effect for calls queued
 * after it, from the pool's one host thread.  Errors: EINVAL.
 */
int kv_pool_set_split_keys(kvx_pool *pool, int32_t keys);

/*
 * Scaled-Q softmax of extend_attention's prefill launches on a bf16 pool (0 =
 * off, the default; 1 = on).  When on, each query is multiplied by
 * c = float32(sm_scale * float32(log2 e)) in float32 and rounded to bf16 (round to
 * nearest even) when it is loaded, and the scores of those queries are taken in
 * base 2: o = softmax_j(ln 2 * bf16(q * c) . k_j) v_j.  This removes one VALU
 * instruction per (query, key) pair, about 5% of the kernel time on long key
 * ranges, and adds one more bf16 rounding of q (2^-9 relative per element): the
 * error against the exact attention grows where scores are large (about twice
 * the default's at query scale 4).  The prefill kernel of an fp8 pool always takes
 * this form (its e4m3 keys dominate the error), and decode steps are always
 * exact.  The softmax itself (Section 2's prefill over the uncached suffix) is
 * unchanged.  A setting of the pool: takes effect for calls queued after it, from
 * the pool's one host thread.  Errors: EINVAL (pool NULL, enable not 0 or 1).
 */
int kv_pool_set_scaled_q(kvx_pool *pool, int32_t enable);

/* Message describing the last non-OK status on this thread ("" if none). */
const char *kvx_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVX_H */
