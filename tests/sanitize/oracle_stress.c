/*
 * Stress of the C oracle (oracle/oracle.c), built with AddressSanitizer and
 * UndefinedBehaviorSanitizer by tests/test_sanitizers.py.
 *
 * Seeded random ragged batches (empty suffixes, unaligned prefixes, several GQA
 * groups, bf16 and fp8 pools) are stored through oracle_store_kv into pools whose
 * every byte starts as a NaN pattern, and every suffix row is attended with
 * oracle_extend_attention.  Outputs must be finite: a read of a slot the batch
 * never wrote would bring a NaN in.  The fp8 codec arrays run over all inputs.
 * Any failure, or any sanitizer report, ends the run with a nonzero status.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_store_kv(int32_t num_reqs, const int32_t *prefix_lens, const int32_t *extend_lens,
                    const int64_t *qo_indptr, const int64_t *page_indptr, const int32_t *page_ids,
                    int32_t page_size, int64_t num_pages, int32_t num_kv_heads, int32_t head_dim,
                    int32_t kv_dtype, const float *k_scale, const float *v_scale,
                    const uint16_t *k_ext, const uint16_t *v_ext, void *k_pool, void *v_pool);
int oracle_extend_attention(int32_t num_reqs, const int32_t *prefix_lens, const int32_t *extend_lens,
                            const int64_t *page_indptr, const int32_t *page_ids, int32_t page_size,
                            int64_t num_pages, int32_t num_q_heads, int32_t num_kv_heads,
                            int32_t head_dim, int32_t kv_dtype, const void *k_pool, const void *v_pool,
                            const float *k_scale, const float *v_scale, int64_t n_rows,
                            const int32_t *row_req, const int32_t *row_pos, const uint16_t *q,
                            double sm_scale, double *out, double *lse, int32_t mutant,
                            int32_t num_threads);
void oracle_e4m3_encode_array(const float *x, int64_t n, uint8_t *out);
void oracle_e4m3_decode_array(const uint8_t *codes, int64_t n, double *out);
uint16_t oracle_bf16_round(double x);

#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            exit(3);                                                       \
        }                                                                  \
    } while (0)

static uint64_t rng_state;
static uint64_t next_u64(void)
{
    /* splitmix64 */
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
static int uni(int lo, int hi) { return lo + (int)(next_u64() % (uint64_t)(hi - lo + 1)); }
static double gauss(void)
{
    double u = ((double)(next_u64() >> 11) + 0.5) / 9007199254740992.0;
    double v = ((double)(next_u64() >> 11) + 0.5) / 9007199254740992.0;
    return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

static void one_batch(int fp8)
{
    const int page = 16;
    int R = uni(1, 5), hkv = uni(1, 3), g = uni(1, 4), d = 8 * uni(1, 4);
    int hq = hkv * g;
    int32_t P[5], E[5];
    int64_t qo[6], indptr[6];
    qo[0] = 0;
    indptr[0] = 0;
    for (int r = 0; r < R; r++) {
        P[r] = uni(0, 90);
        E[r] = uni(0, 3) == 0 ? 0 : uni(1, 50);
        qo[r + 1] = qo[r] + E[r];
        indptr[r + 1] = indptr[r] + (P[r] + E[r] + page - 1) / page;
    }
    int64_t need = indptr[R], num_pages = need + uni(0, 5);
    if (num_pages == 0) num_pages = 1;
    int32_t *ids = malloc(sizeof(int32_t) * (size_t)(need + 1));
    int32_t *perm = malloc(sizeof(int32_t) * (size_t)num_pages);
    for (int64_t i = 0; i < num_pages; i++) perm[i] = (int32_t)i;
    for (int64_t i = num_pages - 1; i > 0; i--) {
        int64_t j = (int64_t)(next_u64() % (uint64_t)(i + 1));
        int32_t t = perm[i];
        perm[i] = perm[j];
        perm[j] = t;
    }
    for (int64_t i = 0; i < need; i++) ids[i] = perm[i];
    /* the whole logical sequence of each request is stored: history rows, then suffix */
    int64_t T = qo[R], L = 0;
    int32_t P0[5], E0[5];
    int64_t qo0[6];
    qo0[0] = 0;
    for (int r = 0; r < R; r++) {
        P0[r] = 0;
        E0[r] = P[r] + E[r];
        qo0[r + 1] = qo0[r] + E0[r];
        L += E0[r];
    }
    size_t row = (size_t)hkv * (size_t)d;
    uint16_t *k = malloc(sizeof(uint16_t) * (size_t)(L + 1) * row);
    uint16_t *v = malloc(sizeof(uint16_t) * (size_t)(L + 1) * row);
    for (size_t i = 0; i < (size_t)L * row; i++) {
        k[i] = oracle_bf16_round(gauss());
        v[i] = oracle_bf16_round(gauss());
    }
    float ks[3], vs[3];
    for (int h = 0; h < hkv; h++) {
        ks[h] = 0.01f + 0.09f * (float)uni(0, 1000) / 1000.0f;
        vs[h] = 0.01f + 0.09f * (float)uni(0, 1000) / 1000.0f;
    }
    size_t eb = fp8 ? 1 : 2;
    size_t pool_bytes = (size_t)num_pages * (size_t)page * row * eb;
    unsigned char *kp = malloc(pool_bytes), *vp = malloc(pool_bytes);
    memset(kp, 0xFF, pool_bytes); /* NaN in bf16 and in e4m3 */
    memset(vp, 0xFF, pool_bytes);
    CHECK(oracle_store_kv(R, P0, E0, qo0, indptr, ids, page, num_pages, hkv, d, fp8, ks, vs, k, v, kp, vp) == 0);
    int32_t *row_req = malloc(sizeof(int32_t) * (size_t)(T + 1));
    int32_t *row_pos = malloc(sizeof(int32_t) * (size_t)(T + 1));
    for (int r = 0; r < R; r++)
        for (int i = 0; i < E[r]; i++) {
            row_req[qo[r] + i] = r;
            row_pos[qo[r] + i] = i;
        }
    uint16_t *q = malloc(sizeof(uint16_t) * (size_t)(T + 1) * (size_t)hq * (size_t)d);
    for (size_t i = 0; i < (size_t)T * (size_t)hq * (size_t)d; i++) q[i] = oracle_bf16_round(gauss());
    double *out = malloc(sizeof(double) * (size_t)(T + 1) * (size_t)hq * (size_t)d);
    double *lse = malloc(sizeof(double) * (size_t)(T + 1) * (size_t)hq);
    CHECK(oracle_extend_attention(R, P, E, indptr, ids, page, num_pages, hq, hkv, d, fp8, kp, vp, ks, vs, T,
                                  row_req, row_pos, q, 1.0 / sqrt((double)d), out, lse, 0, 2) == 0);
    for (size_t i = 0; i < (size_t)T * (size_t)hq * (size_t)d; i++) CHECK(isfinite(out[i]));
    for (size_t i = 0; i < (size_t)T * (size_t)hq; i++) CHECK(isfinite(lse[i]));
    /* a row outside its request is refused */
    if (T > 0) {
        int32_t bad = E[row_req[0]];
        CHECK(oracle_extend_attention(R, P, E, indptr, ids, page, num_pages, hq, hkv, d, fp8, kp, vp, ks, vs, 1,
                                      row_req, &bad, q, 0.125, out, NULL, 0, 1) == -1);
    }
    free(ids);
    free(perm);
    free(k);
    free(v);
    free(kp);
    free(vp);
    free(row_req);
    free(row_pos);
    free(q);
    free(out);
    free(lse);
}

int main(int argc, char **argv)
{
    int n = argc > 1 ? atoi(argv[1]) : 200;
    rng_state = 12345;
    for (int i = 0; i < n; i++) one_batch(i % 3 == 2);
    /* the e4m3 codec over every bf16 input */
    float *x = malloc(sizeof(float) * 65536);
    uint8_t *c = malloc(65536);
    double *back = malloc(sizeof(double) * 65536);
    for (uint32_t b = 0; b < 65536; b++) {
        uint32_t w = b << 16;
        memcpy(&x[b], &w, 4);
    }
    oracle_e4m3_encode_array(x, 65536, c);
    oracle_e4m3_decode_array(c, 65536, back);
    free(x);
    free(c);
    free(back);
    printf("oracle stress: %d batches passed\n", n);
    return 0;
}
