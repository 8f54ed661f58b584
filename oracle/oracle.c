/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct fp64 CPU oracle of prefix-extend attention
 * over a paged KV pool.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load it; the product path never calls it, and it shares no
 * code, header, table or helper with the HIP library.
 *
 * What it computes.  A returning agent reuses the KV tensors of its cached
 * prefix and computes only the uncached suffix (Section 1; Section 2, "Prefix
 * caching for multi-turn agents").  Reuse does not change the result: every
 * suffix query at absolute position t attends, with a softmax, over the keys
 * at positions 0..t of the request's logical token sequence, whether those
 * keys come from the cached prefix or from the suffix itself.  The suffix's
 * K/V are first written into the pool (prefill materialises KV in every
 * attention layer, Section 2).  The oracle is that definition written out:
 *
 *   oracle_store_kv:        pool[page_of(P+i)][h][(P+i) % S][:] = K_ext[row][h][:]
 *   oracle_store_kv_f64:    the same placement for K given as exact values
 *                            (the rotated keys of the RoPE store, oracle/rope.py),
 *                            rounded once into the pool's format
 *   oracle_extend_attention: s_j = scale * <q, k_j>, w_j = exp(s_j - max s),
 *                            o = sum_j w_j v_j / sum_j w_j,  lse = max s + ln(sum w)
 *
 * Readings where the paper is silent (it describes no kernel arithmetic):
 *   - GQA: query head hq uses KV head hq / (Hq / Hkv).
 *   - Causality is aligned bottom-right and inclusive: suffix row i of a request
 *     with prefix P sees keys 0..P+i.
 *   - Pool layout is [page][kv_head][slot][head_dim] for both K and V.
 *   - fp8 pool: OCP E4M3 ("e4m3fn": bias 7, no infinities, 0x7F/0xFF are NaN,
 *     largest finite 448).  A stored code is
 *        encode( float(x) * float(1/scale) )
 *     computed in fp32, rounded to nearest with ties to even, saturating at
 *     +-448; the attention reads decode(code) * scale.
 *
 * Precision: all attention arithmetic is in double.  bf16 and e4m3 inputs are
 * exactly representable in double.
 */

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_KV_BF16 0
#define ORACLE_KV_FP8_E4M3 1

/* Planted mistakes, used only by tests that show the parity gate and the pins
 * can tell a wrong implementation from the right one (0 = the oracle itself). */
#define MUT_NONE 0
#define MUT_EXCLUSIVE_DIAGONAL 1  /* row sees keys 0..t-1 */
#define MUT_TOP_LEFT_CAUSAL 2     /* row i sees keys 0..i (prefix offset ignored) */
#define MUT_KV_HEAD_MODULO 3      /* kv head = hq % Hkv */
#define MUT_DROP_PARTIAL_PAGE 4   /* keys of a partially filled last page ignored */
#define MUT_IGNORE_PREFIX 5       /* keys of the cached prefix ignored */
#define MUT_REVERSED_PAGES 6      /* logical page j read from the table's other end */
#define MUT_SCALE_ONE_OVER_D 7    /* softmax scale 1/d instead of the given one */

/* ------------------------------------------------------------------ number formats */

double oracle_bf16_to_double(uint16_t bits)
{
    /* bf16 is the upper half of an IEEE binary32 */
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static float bf16_to_float(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* The bf16 value nearest to a double, ties to the even significand: bf16 keeps
 * 8 significant bits (7 stored) over binary32's exponent range, so the
 * quantum of |x| in [2^(e-1), 2^e) is 2^(e-8), and 2^-133 below the smallest
 * normal 2^-126.  Rounding straight from the double (not through a float)
 * avoids a second rounding.  Magnitudes past the largest finite bf16 round to
 * infinity the way binary32 overflow does. */
uint16_t oracle_bf16_round(double x)
{
    if (isnan(x))
        return 0x7FC0;
    double a = fabs(x);
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    if (a == 0.0)
        return sign;
    int e;
    frexp(a, &e);
    int q = e - 8;
    if (q < -133)
        q = -133;
    double r = ldexp(nearbyint(ldexp(a, -q)), q); /* default rounding: ties to even */
    float f = (float)r;                            /* exact, or inf past the range */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(sign | (uint16_t)((u >> 16) & 0x7FFF));
}

void oracle_bf16_round_array(const double *x, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_bf16_round(x[i]);
}

/* OCP 8-bit floating point, E4M3 variant: 1 sign bit, 4 exponent bits (bias 7),
 * 3 mantissa bits.  Exponent field 0 encodes subnormals m/8 * 2^-6; the pattern
 * with all exponent and mantissa bits set is NaN; there is no infinity. */
double oracle_e4m3_decode(uint8_t code)
{
    int sign = (code >> 7) & 1;
    int e = (code >> 3) & 0xF;
    int m = code & 0x7;
    double mag;
    if (e == 0xF && m == 0x7)
        return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, -6);
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -mag : mag;
}

/* The 127 non-negative finite magnitudes in code order (codes 0x00..0x7E are
 * increasing), filled from the decoder above. */
static double e4m3_mag[127];
static int e4m3_mag_ready = 0;

static void e4m3_table_init(void)
{
    if (e4m3_mag_ready)
        return;
    for (int c = 0; c <= 0x7E; c++)
        e4m3_mag[c] = oracle_e4m3_decode((uint8_t)c);
    e4m3_mag_ready = 1;
}

/* Encode: the nearest non-negative finite code to |x|, ties to the code with an
 * even mantissa (= the even code), magnitudes above the largest finite value
 * saturate to it; then the sign bit.  The table must be initialised. */
static uint8_t e4m3_encode_nearest(float x)
{
    if (isnan(x))
        return 0x7F;
    int neg = signbit(x) ? 1 : 0;
    double a = fabs((double)x);
    int best;
    if (a >= e4m3_mag[0x7E]) {
        best = 0x7E; /* saturate */
    } else {
        /* largest lo with mag[lo] <= a < mag[lo + 1] */
        int lo = 0, hi = 0x7E;
        while (hi - lo > 1) {
            int mid = (lo + hi) / 2;
            if (e4m3_mag[mid] <= a)
                lo = mid;
            else
                hi = mid;
        }
        double below = a - e4m3_mag[lo], above = e4m3_mag[hi] - a;
        if (below < above)
            best = lo;
        else if (above < below)
            best = hi;
        else
            best = (lo % 2 == 0) ? lo : hi;
    }
    return (uint8_t)((neg << 7) | best);
}

uint8_t oracle_e4m3_encode(float x)
{
    e4m3_table_init();
    return e4m3_encode_nearest(x);
}

void oracle_e4m3_encode_array(const float *x, int64_t n, uint8_t *out)
{
    e4m3_table_init();
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_e4m3_encode(x[i]);
}

void oracle_e4m3_decode_array(const uint8_t *codes, int64_t n, double *out)
{
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_e4m3_decode(codes[i]);
}

/* ------------------------------------------------------------------------ KV store */

static int64_t pool_offset(int64_t page, int h, int slot, int c, int num_kv_heads, int page_size,
                           int head_dim)
{
    return (((page * num_kv_heads) + h) * page_size + slot) * (int64_t)head_dim + c;
}

/* Write every suffix token's K and V rows into the request's pages.  K comes
 * either as bf16 bits (k_bits) or as exact real values (k_vals, double; the
 * rotated keys of the RoPE store): a bf16 pool holds bf16 bits, rounded to
 * nearest-even from the double when k_vals is given; an fp8 pool holds
 * encode(float(x) * float(1/scale)).  V always comes as bf16 bits.  Returns 0,
 * or -1 if a page id falls outside [0, num_pages) (those tokens are skipped).
 * Suffix tokens map to distinct (page, slot) pairs in a valid batch, so the
 * per-token loop may run in parallel. */
static int store_rows(int32_t num_reqs, const int32_t *prefix_lens, const int32_t *extend_lens,
                      const int64_t *qo_indptr, const int64_t *page_indptr, const int32_t *page_ids,
                      int32_t page_size, int64_t num_pages, int32_t num_kv_heads, int32_t head_dim,
                      int32_t kv_dtype, const float *k_scale, const float *v_scale,
                      const uint16_t *k_bits, const double *k_vals, const uint16_t *v_ext,
                      void *k_pool, void *v_pool)
{
    int status = 0;
    e4m3_table_init();
    for (int r = 0; r < num_reqs; r++) {
#pragma omp parallel for schedule(static)
        for (int i = 0; i < extend_lens[r]; i++) {
            int64_t t = (int64_t)prefix_lens[r] + i;
            int64_t page = page_ids[page_indptr[r] + t / page_size];
            int slot = (int)(t % page_size);
            int64_t row = qo_indptr[r] + i;
            if (page < 0 || page >= num_pages) {
#pragma omp atomic write
                status = -1;
                continue;
            }
            for (int h = 0; h < num_kv_heads; h++) {
                for (int c = 0; c < head_dim; c++) {
                    int64_t src = (row * num_kv_heads + h) * (int64_t)head_dim + c;
                    int64_t dst = pool_offset(page, h, slot, c, num_kv_heads, page_size, head_dim);
                    if (kv_dtype == ORACLE_KV_BF16) {
                        ((uint16_t *)k_pool)[dst] = k_vals ? oracle_bf16_round(k_vals[src]) : k_bits[src];
                        ((uint16_t *)v_pool)[dst] = v_ext[src];
                    } else {
                        float kinv = 1.0f / k_scale[h];
                        float vinv = 1.0f / v_scale[h];
                        float k = k_vals ? (float)k_vals[src] : bf16_to_float(k_bits[src]);
                        float kx = k * kinv;
                        float vx = bf16_to_float(v_ext[src]) * vinv;
                        ((uint8_t *)k_pool)[dst] = e4m3_encode_nearest(kx);
                        ((uint8_t *)v_pool)[dst] = e4m3_encode_nearest(vx);
                    }
                }
            }
        }
    }
    return status;
}

int oracle_store_kv(int32_t num_reqs, const int32_t *prefix_lens, const int32_t *extend_lens,
                    const int64_t *qo_indptr, const int64_t *page_indptr, const int32_t *page_ids,
                    int32_t page_size, int64_t num_pages, int32_t num_kv_heads, int32_t head_dim,
                    int32_t kv_dtype, const float *k_scale, const float *v_scale,
                    const uint16_t *k_ext, const uint16_t *v_ext, void *k_pool, void *v_pool)
{
    return store_rows(num_reqs, prefix_lens, extend_lens, qo_indptr, page_indptr, page_ids, page_size,
                      num_pages, num_kv_heads, head_dim, kv_dtype, k_scale, v_scale, k_ext, NULL, v_ext,
                      k_pool, v_pool);
}

/* The same store with K given as doubles (see store_rows). */
int oracle_store_kv_f64(int32_t num_reqs, const int32_t *prefix_lens, const int32_t *extend_lens,
                        const int64_t *qo_indptr, const int64_t *page_indptr, const int32_t *page_ids,
                        int32_t page_size, int64_t num_pages, int32_t num_kv_heads, int32_t head_dim,
                        int32_t kv_dtype, const float *k_scale, const float *v_scale,
                        const double *k_vals, const uint16_t *v_ext, void *k_pool, void *v_pool)
{
    return store_rows(num_reqs, prefix_lens, extend_lens, qo_indptr, page_indptr, page_ids, page_size,
                      num_pages, num_kv_heads, head_dim, kv_dtype, k_scale, v_scale, NULL, k_vals, v_ext,
                      k_pool, v_pool);
}

/* ------------------------------------------------------------------- attention */

static double pool_value(const void *pool, int32_t kv_dtype, const float *scale, int64_t off, int h)
{
    if (kv_dtype == ORACLE_KV_BF16)
        return oracle_bf16_to_double(((const uint16_t *)pool)[off]);
    return oracle_e4m3_decode(((const uint8_t *)pool)[off]) * (double)scale[h];
}

/*
 * Attention for an explicit list of suffix rows: row n is suffix position
 * row_pos[n] of request row_req[n]; its queries are q[n][0..Hq)[0..d) (bf16
 * bits) and its outputs go to out[n][hq][c] (and lse[n][hq] if lse != NULL).
 * Returns 0, or -1 on a page id outside the pool / a row outside its request.
 */
int oracle_extend_attention(int32_t num_reqs, const int32_t *prefix_lens, const int32_t *extend_lens,
                            const int64_t *page_indptr, const int32_t *page_ids, int32_t page_size,
                            int64_t num_pages, int32_t num_q_heads, int32_t num_kv_heads,
                            int32_t head_dim, int32_t kv_dtype, const void *k_pool, const void *v_pool,
                            const float *k_scale, const float *v_scale, int64_t n_rows,
                            const int32_t *row_req, const int32_t *row_pos, const uint16_t *q,
                            double sm_scale, double *out, double *lse, int32_t mutant,
                            int32_t num_threads)
{
    int group = num_q_heads / num_kv_heads;
    int64_t tasks = n_rows * num_q_heads;
    int status = 0;
    for (int64_t n = 0; n < n_rows; n++) {
        int r = row_req[n];
        if (r < 0 || r >= num_reqs || row_pos[n] < 0 || row_pos[n] >= extend_lens[r])
            return -1;
    }
#ifdef _OPENMP
    if (num_threads > 0)
        omp_set_num_threads(num_threads);
#else
    (void)num_threads;
#endif

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t task = 0; task < tasks; task++) {
        int64_t n = task / num_q_heads;
        int hq = (int)(task % num_q_heads);
        int r = row_req[n];
        int64_t P = prefix_lens[r];
        int64_t L = P + extend_lens[r];
        int64_t i = row_pos[n];
        int64_t t = P + i;
        int64_t n_pages = page_indptr[r + 1] - page_indptr[r];
        int h = (mutant == MUT_KV_HEAD_MODULO) ? hq % num_kv_heads : hq / group;
        double scale = sm_scale;
        if (mutant == MUT_SCALE_ONE_OVER_D)
            scale = 1.0 / (double)head_dim;

        /* visible keys [lo, hi] */
        int64_t lo = 0, hi = t;
        if (mutant == MUT_EXCLUSIVE_DIAGONAL)
            hi = t - 1;
        if (mutant == MUT_TOP_LEFT_CAUSAL)
            hi = i;
        if (mutant == MUT_IGNORE_PREFIX)
            lo = P;
        if (mutant == MUT_DROP_PARTIAL_PAGE && (L % page_size) != 0) {
            int64_t full = (L / page_size) * page_size;
            if (hi > full - 1)
                hi = full - 1;
        }

        const uint16_t *qrow = q + (n * num_q_heads + hq) * (int64_t)head_dim;
        double *o = out + (n * num_q_heads + hq) * (int64_t)head_dim;
        for (int c = 0; c < head_dim; c++)
            o[c] = 0.0;
        if (hi < lo) {
            if (lse)
                lse[n * num_q_heads + hq] = -INFINITY;
            continue;
        }

        int64_t nk = hi - lo + 1;
        double *s = (double *)malloc(sizeof(double) * (size_t)nk);
        int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)nk);
        if (!s || !off) {
            free(s);
            free(off);
#pragma omp atomic write
            status = -2;
            continue;
        }
        int bad = 0;
        for (int64_t j = lo; j <= hi; j++) {
            int64_t lp = j / page_size;
            if (mutant == MUT_REVERSED_PAGES)
                lp = n_pages - 1 - lp;
            int64_t page = page_ids[page_indptr[r] + lp];
            if (page < 0 || page >= num_pages) {
                bad = 1;
                break;
            }
            off[j - lo] = pool_offset(page, h, (int)(j % page_size), 0, num_kv_heads, page_size,
                                      head_dim);
        }
        if (bad) {
            free(s);
            free(off);
#pragma omp atomic write
            status = -1;
            continue;
        }

        /* scores and their maximum */
        double m = -INFINITY;
        for (int64_t j = 0; j < nk; j++) {
            double dot = 0.0;
            for (int c = 0; c < head_dim; c++)
                dot += oracle_bf16_to_double(qrow[c]) *
                       pool_value(k_pool, kv_dtype, k_scale, off[j] + c, h);
            s[j] = scale * dot;
            if (s[j] > m)
                m = s[j];
        }
        /* softmax weights and the weighted sum of values */
        double z = 0.0;
        for (int64_t j = 0; j < nk; j++) {
            double w = exp(s[j] - m);
            z += w;
            for (int c = 0; c < head_dim; c++)
                o[c] += w * pool_value(v_pool, kv_dtype, v_scale, off[j] + c, h);
        }
        for (int c = 0; c < head_dim; c++)
            o[c] /= z;
        if (lse)
            lse[n * num_q_heads + hq] = m + log(z);
        free(s);
        free(off);
    }
    return status;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
