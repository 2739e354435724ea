/*
 * fp64 CPU oracle for fused scaled-dot-product attention forward.
 *
 * TEST INFRASTRUCTURE: this file is the reference the GPU path is checked
 * against.  Only the test suite, the smoke check and the bench's CPU-baseline
 * leg may load it; the product path never calls it, and it shares no code,
 * header, table or helper with the HIP library.
 *
 * What it computes is the plain definition that the tiled online-softmax
 * recurrence of the paper's attention kernel reaches in exact arithmetic
 * (paper, Appendix "Implementation of FlashMLA with TileLang": running max,
 * rescale by exp of the max difference, running sum, final division by the
 * sum).  Because that recurrence is exact up to rounding order, the oracle is
 * the definition itself, written out one output row at a time:
 *
 *   for batch b, query head h, query row i:
 *     g  = Hq / Hkv,  hk = floor(h / g)          (grouped-query head map)
 *     n  = Sk                      if not causal
 *        = min(Sk, i + 1 + Sk-Sq)  if causal      (bottom-right alignment:
 *                                                   key j visible iff
 *                                                   j <= i + Sk - Sq)
 *     s_j = scale * sum_d Q[b,h,i,d] * K[b,hk,j,d]            for j < n
 *     m   = max_j s_j
 *     z   = sum_j exp(s_j - m)
 *     LSE[b,h,i] = m + ln z          (natural log of sum_j exp(s_j))
 *     O[b,h,i,d] = sum_j exp(s_j - m) * V[b,hk,j,d] / z
 *
 * There are no tiles, no running max and no base-2 exponentials.  Inputs are
 * bfloat16 bit patterns (widened exactly); every operation is in double
 * precision with plain ascending loops.  Tensors are contiguous BHSD:
 * Q, O [B,Hq,Sq,D]; K, V [B,Hkv,Sk,D]; LSE [B,Hq,Sq].
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    const uint16_t *Q, *K, *V;
    int64_t B, Hq, Hkv, Sq, Sk, D;
    int causal;
    double scale;
} problem;

/* bfloat16 bits -> double, exactly: a bfloat16 is the top half of a float. */
static double widen(uint16_t bits)
{
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* Number of keys query row i may attend to. */
static int64_t visible_keys(const problem *p, int64_t i)
{
    if (!p->causal)
        return p->Sk;
    int64_t n = i + 1 + (p->Sk - p->Sq);
    return n < p->Sk ? n : p->Sk;
}

/* One output row (b, h, i).  s is scratch of length Sk. */
static void attend_row(const problem *p, int64_t b, int64_t h, int64_t i,
                       double *s, double *o, double *lse)
{
    const int64_t D = p->D;
    const int64_t hk = h / (p->Hq / p->Hkv);
    const uint16_t *q = p->Q + ((b * p->Hq + h) * p->Sq + i) * D;
    const uint16_t *k = p->K + (b * p->Hkv + hk) * p->Sk * D;
    const uint16_t *v = p->V + (b * p->Hkv + hk) * p->Sk * D;
    const int64_t n = visible_keys(p, i);

    for (int64_t j = 0; j < n; ++j) {
        double dot = 0.0;
        for (int64_t d = 0; d < D; ++d)
            dot += widen(q[d]) * widen(k[j * D + d]);
        s[j] = p->scale * dot;
    }

    double m = -INFINITY;
    for (int64_t j = 0; j < n; ++j)
        if (s[j] > m)
            m = s[j];

    double z = 0.0;
    for (int64_t j = 0; j < n; ++j)
        z += exp(s[j] - m);
    *lse = m + log(z);

    for (int64_t d = 0; d < D; ++d)
        o[d] = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        const double w = exp(s[j] - m);
        for (int64_t d = 0; d < D; ++d)
            o[d] += w * widen(v[j * D + d]);
    }
    for (int64_t d = 0; d < D; ++d)
        o[d] /= z;
}

/* Shape rules shared by both entry points; 0 = valid. */
static int check(const problem *p)
{
    if (!p->Q || !p->K || !p->V)
        return 1;
    if (p->B < 1 || p->Hq < 1 || p->Hkv < 1 || p->Sq < 1 || p->Sk < 1 || p->D < 1)
        return 2;
    if (p->Hq % p->Hkv != 0)
        return 2;
    if (p->causal && p->Sq > p->Sk)
        return 2;
    return 0;
}

/* ---- threading: rows are independent, split them evenly ---------------- */

typedef struct {
    const problem *p;
    const int64_t *rows;   /* NULL: every row, row r = ((b*Hq)+h)*Sq + i */
    int64_t first, last;   /* half-open range of work items */
    double *O, *LSE;
    int failed;
} job;

static void *run_job(void *arg)
{
    job *jb = (job *)arg;
    const problem *p = jb->p;
    double *s = (double *)malloc(sizeof(double) * (size_t)p->Sk);
    if (!s) {
        jb->failed = 1;
        return NULL;
    }
    for (int64_t r = jb->first; r < jb->last; ++r) {
        int64_t b, h, i;
        if (jb->rows) {
            b = jb->rows[3 * r];
            h = jb->rows[3 * r + 1];
            i = jb->rows[3 * r + 2];
        } else {
            i = r % p->Sq;
            h = (r / p->Sq) % p->Hq;
            b = r / (p->Sq * p->Hq);
        }
        attend_row(p, b, h, i, s, jb->O + r * p->D, jb->LSE + r);
    }
    free(s);
    return NULL;
}

static int run(const problem *p, const int64_t *rows, int64_t nrows,
               double *O, double *LSE, int nthreads)
{
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > 256)
        nthreads = 256;
    if ((int64_t)nthreads > nrows)
        nthreads = (int)nrows;
    pthread_t tid[256];
    int spawned[256];
    job jobs[256];
    int rc = 0;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = (job){p, rows, nrows * t / nthreads, nrows * (t + 1) / nthreads, O, LSE, 0};
        /* the last slice, and any slice whose thread fails to start, runs here */
        spawned[t] = t < nthreads - 1 && pthread_create(&tid[t], NULL, run_job, &jobs[t]) == 0;
        if (!spawned[t])
            run_job(&jobs[t]);
    }
    for (int t = 0; t < nthreads; ++t) {
        if (spawned[t])
            pthread_join(tid[t], NULL);
        rc |= jobs[t].failed;
    }
    return rc ? 3 : 0;
}

/*
 * Every output row.  O: [B,Hq,Sq,D] doubles, LSE: [B,Hq,Sq] doubles.
 * Returns 0, or 1 (null input), 2 (invalid shape), 3 (out of memory).
 */
int oracle_attn_fwd(const uint16_t *Q, const uint16_t *K, const uint16_t *V,
                    double *O, double *LSE,
                    int64_t B, int64_t Hq, int64_t Hkv, int64_t Sq, int64_t Sk, int64_t D,
                    int causal, double scale, int nthreads)
{
    problem p = {Q, K, V, B, Hq, Hkv, Sq, Sk, D, causal, scale};
    int rc = check(&p);
    if (rc)
        return rc;
    if (!O || !LSE)
        return 1;
    return run(&p, NULL, B * Hq * Sq, O, LSE, nthreads);
}

/*
 * Selected rows only: rows is [nrows][3] of (b, h, i).  O: [nrows, D],
 * LSE: [nrows].  Same return codes; 2 also for a row index out of range.
 */
int oracle_attn_rows(const uint16_t *Q, const uint16_t *K, const uint16_t *V,
                     int64_t B, int64_t Hq, int64_t Hkv, int64_t Sq, int64_t Sk, int64_t D,
                     int causal, double scale,
                     const int64_t *rows, int64_t nrows, double *O, double *LSE, int nthreads)
{
    problem p = {Q, K, V, B, Hq, Hkv, Sq, Sk, D, causal, scale};
    int rc = check(&p);
    if (rc)
        return rc;
    if (!rows || !O || !LSE)
        return 1;
    for (int64_t r = 0; r < nrows; ++r)
        if (rows[3 * r] < 0 || rows[3 * r] >= B || rows[3 * r + 1] < 0 || rows[3 * r + 1] >= Hq ||
            rows[3 * r + 2] < 0 || rows[3 * r + 2] >= Sq)
            return 2;
    if (nrows == 0)
        return 0;
    return run(&p, rows, nrows, O, LSE, nthreads);
}
