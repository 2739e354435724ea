/*
 * The fp64 attention oracle (oracle/attn_oracle.c) built with
 * AddressSanitizer and UndefinedBehaviorSanitizer and run on small problems
 * of every kind it accepts (tests/test_sanitizers.py builds and runs it on
 * the CPU): non-causal and bottom-right causal, grouped-query heads, one
 * query or one key, query and key lengths that differ, head dims 4, 64 and
 * 128, single- and multi-threaded, every row and selected rows.  Besides
 * any sanitizer report, it fails on an error status, a non-finite output, an
 * output row outside the range of the value rows (each is a weighted mean of
 * them), a causal row 0 that is not value row 0, or a selected-rows result
 * that differs from the every-row result.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_attn_fwd(const uint16_t *Q, const uint16_t *K, const uint16_t *V, double *O,
                    double *LSE, int64_t B, int64_t Hq, int64_t Hkv, int64_t Sq, int64_t Sk,
                    int64_t D, int causal, double scale, int nthreads);
int oracle_attn_rows(const uint16_t *Q, const uint16_t *K, const uint16_t *V, int64_t B,
                     int64_t Hq, int64_t Hkv, int64_t Sq, int64_t Sk, int64_t D, int causal,
                     double scale, const int64_t *rows, int64_t nrows, double *O, double *LSE,
                     int nthreads);

static int failures = 0;
static uint64_t rng = 88172645463325252ull;

static uint16_t rand_bf16(void)
{
    /* xorshift64, mapped to a float in [-2, 2), truncated to bfloat16 */
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    float f = (float)((rng >> 11) * (1.0 / 9007199254740992.0)) * 4.0f - 2.0f;
    uint32_t w;
    memcpy(&w, &f, sizeof w);
    return (uint16_t)(w >> 16);
}

static double wide(uint16_t b)
{
    uint32_t w = (uint32_t)b << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return f;
}

static void one(int64_t B, int64_t Hq, int64_t Hkv, int64_t Sq, int64_t Sk, int64_t D,
                int causal, int threads)
{
    const size_t nq = (size_t)(B * Hq * Sq * D), nkv = (size_t)(B * Hkv * Sk * D);
    uint16_t *q = malloc(nq * 2), *k = malloc(nkv * 2), *v = malloc(nkv * 2);
    double *o = malloc(nq * 8), *l = malloc((size_t)(B * Hq * Sq) * 8);
    for (size_t i = 0; i < nq; ++i)
        q[i] = rand_bf16();
    for (size_t i = 0; i < nkv; ++i) {
        k[i] = rand_bf16();
        v[i] = rand_bf16();
    }
    const double scale = 1.0 / sqrt((double)D);
    int rc = oracle_attn_fwd(q, k, v, o, l, B, Hq, Hkv, Sq, Sk, D, causal, scale, threads);
    if (rc != 0) {
        fprintf(stderr, "FAIL status %d for B%lld Hq%lld Hkv%lld Sq%lld Sk%lld D%lld c%d\n", rc,
                (long long)B, (long long)Hq, (long long)Hkv, (long long)Sq, (long long)Sk,
                (long long)D, causal);
        ++failures;
        goto out;
    }
    const int64_t g = Hq / Hkv;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t h = 0; h < Hq; ++h)
            for (int64_t i = 0; i < Sq; ++i) {
                const size_t r = (size_t)((b * Hq + h) * Sq + i);
                const int64_t n = causal ? (i + 1 + Sk - Sq < Sk ? i + 1 + Sk - Sq : Sk) : Sk;
                if (!isfinite(l[r]))
                    ++failures;
                for (int64_t d = 0; d < D; ++d) {
                    double lo = INFINITY, hi = -INFINITY;
                    for (int64_t j = 0; j < n; ++j) {
                        const double x = wide(v[(size_t)(((b * Hkv + h / g) * Sk + j) * D + d)]);
                        lo = x < lo ? x : lo;
                        hi = x > hi ? x : hi;
                    }
                    const double y = o[r * (size_t)D + (size_t)d];
                    if (!(isfinite(y) && y >= lo - 1e-12 && y <= hi + 1e-12)) {
                        fprintf(stderr, "FAIL O outside the V range at row %zu d %lld\n", r,
                                (long long)d);
                        ++failures;
                    }
                    if (causal && Sq == Sk && i == 0 &&
                        y != wide(v[(size_t)((b * Hkv + h / g) * Sk * D + d)])) {
                        fprintf(stderr, "FAIL causal row 0 is not V row 0\n");
                        ++failures;
                    }
                }
            }
    /* the last row of every head through the selected-rows entry */
    {
        const int64_t nr = B * Hq;
        int64_t *rows = malloc((size_t)nr * 3 * sizeof(int64_t));
        double *o2 = malloc((size_t)(nr * D) * 8), *l2 = malloc((size_t)nr * 8);
        for (int64_t x = 0; x < nr; ++x) {
            rows[3 * x] = x / Hq;
            rows[3 * x + 1] = x % Hq;
            rows[3 * x + 2] = Sq - 1;
        }
        rc = oracle_attn_rows(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, scale, rows, nr, o2, l2,
                              threads);
        if (rc != 0)
            ++failures;
        for (int64_t x = 0; x < nr && rc == 0; ++x) {
            const size_t r = (size_t)(x * Sq + Sq - 1);
            if (l2[x] != l[r] || memcmp(o2 + x * D, o + r * (size_t)D, (size_t)D * 8) != 0) {
                fprintf(stderr, "FAIL selected row differs from the every-row result\n");
                ++failures;
            }
        }
        /* an out-of-range row is rejected */
        rows[2] = Sq;
        if (oracle_attn_rows(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, scale, rows, 1, o2, l2,
                             threads) != 2)
            ++failures;
        free(rows);
        free(o2);
        free(l2);
    }
out:
    free(q);
    free(k);
    free(v);
    free(o);
    free(l);
}

int main(void)
{
    const int64_t shapes[][7] = {
        /* B, Hq, Hkv, Sq, Sk, D, causal */
        {1, 1, 1, 1, 1, 4, 0},      {1, 1, 1, 1, 1, 64, 1},    {2, 2, 1, 5, 9, 4, 1},
        {1, 4, 2, 17, 17, 64, 1},   {1, 2, 2, 33, 70, 128, 0}, {2, 3, 1, 7, 7, 4, 0},
        {1, 8, 2, 1, 129, 64, 1},   {1, 2, 2, 65, 65, 128, 1}, {1, 1, 1, 100, 37, 4, 0},
    };
    for (size_t s = 0; s < sizeof shapes / sizeof shapes[0]; ++s)
        for (int threads = 1; threads <= 3; threads += 2)
            one(shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3], shapes[s][4],
                shapes[s][5], (int)shapes[s][6], threads);
    /* invalid arguments are reported, not dereferenced */
    uint16_t x[16] = {0};
    double o[16], l[4];
    if (oracle_attn_fwd(NULL, x, x, o, l, 1, 1, 1, 1, 1, 4, 0, 1.0, 1) != 1)
        ++failures;
    if (oracle_attn_fwd(x, x, x, o, l, 1, 3, 2, 1, 1, 4, 0, 1.0, 1) != 2)
        ++failures;
    if (oracle_attn_fwd(x, x, x, o, l, 1, 1, 1, 2, 1, 4, 1, 1.0, 1) != 2)
        ++failures;
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("oracle_driver: all checks passed\n");
    return 0;
}
