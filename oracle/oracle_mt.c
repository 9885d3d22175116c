/*
 * Multi-core variant of the CPU oracle (TEST INFRASTRUCTURE ONLY), for the
 * timing baseline on all host cores and for checking long error-feedback runs
 * in reasonable time.  It returns exactly what the single-threaded functions
 * of oracle.c return (a CPU test compares them bit for bit); only the work is
 * split into contiguous index chunks, one per OpenMP thread.
 *
 *   orc_ht_mt          the hard threshold is element-wise (section 4.2:
 *                      S_lambda(x) = { i : |x[i]| >= lambda }), so each chunk
 *                      is orc_ht itself on that chunk; a first pass counts
 *                      every chunk's kept coordinates so that each writes its
 *                      pairs at its place in the ascending-index payload.
 *   orc_topk_mt        Top-k (Lemma 2; ties to the lower index): each chunk
 *                      sorts its coordinates by (key descending, index
 *                      ascending), the first k of the merged chunk orders are
 *                      the first k of the whole order, then the pairs are
 *                      written in ascending index order.
 *   orc_topk_segmented_mt  layer-wise Top-k (Appendix C.5): orc_topk on
 *                      each segment, the segments shared out over the threads
 *                      (each segment's payload region is known in advance).
 *   orc_accumulate_mt  the exchange-and-average step: the same in-order sum
 *                      as orc_accumulate, with the zero fill and the division
 *                      by n split over the threads.
 *
 * Built together with oracle.c (it calls orc_ht and orc_topk) with -fopenmp, and with the
 * same floating-point flags: -ffp-contract=off, no fast-math, SSE arithmetic.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

void orc_ht(const float *g, float *e, int64_t d, float lr, float lambda,
            int32_t *idx, float *val, int64_t cap, int64_t *count);
int orc_topk(const float *g, float *e, int64_t d, float lr, int64_t k,
             int32_t *idx, float *val);

int orc_mt_threads(void) { return omp_get_max_threads(); }

/* Chunk c of nc over [0, d): [lo, hi). */
static void chunk_bounds(int64_t d, int nc, int c, int64_t *lo, int64_t *hi)
{
    *lo = d * c / nc;
    *hi = d * (c + 1) / nc;
}

/* p = e + lr*g as two separately rounded fp32 operations (Algorithm 1). */
static float ef_accumulate(float e, float lr, float g)
{
    float scaled = lr * g;
    return e + scaled;
}

void orc_ht_mt(const float *g, float *e, int64_t d, float lr, float lambda,
               int32_t *idx, float *val, int64_t cap, int64_t *count)
{
    const int nc = omp_get_max_threads();
    int64_t *kept = (int64_t *)calloc((size_t)nc + 1, sizeof *kept);
    if (!kept) {  /* no scratch: the single-threaded definition */
        orc_ht(g, e, d, lr, lambda, idx, val, cap, count);
        return;
    }
#pragma omp parallel for schedule(static, 1) num_threads(nc)
    for (int c = 0; c < nc; c++) {
        int64_t lo, hi, n = 0;
        chunk_bounds(d, nc, c, &lo, &hi);
        for (int64_t i = lo; i < hi; i++)
            if (fabsf(ef_accumulate(e[i], lr, g[i])) >= lambda) n++;
        kept[c + 1] = n;
    }
    for (int c = 0; c < nc; c++) kept[c + 1] += kept[c];
#pragma omp parallel for schedule(static, 1) num_threads(nc)
    for (int c = 0; c < nc; c++) {
        int64_t lo, hi, n = 0;
        chunk_bounds(d, nc, c, &lo, &hi);
        const int64_t off = kept[c];
        int64_t room = cap - off;
        if (room < 0) room = 0;
        orc_ht(g + lo, e + lo, hi - lo, lr, lambda, idx + (room ? off : 0),
               val + (room ? off : 0), room, &n);
        const int64_t written = n < room ? n : room;
        for (int64_t j = 0; j < written; j++) idx[off + j] += (int32_t)lo;
    }
    *count = kept[nc];
    free(kept);
}

typedef struct {
    uint32_t key;
    int32_t index;
} mt_rank;

static uint32_t magnitude_key(float p)
{
    uint32_t bits;
    memcpy(&bits, &p, sizeof bits);
    return bits & 0x7fffffffu;
}

/* Larger key first; equal keys by lower index first. */
static int before(const mt_rank *x, const mt_rank *y)
{
    if (x->key != y->key) return x->key > y->key;
    return x->index < y->index;
}

static int rank_cmp(const void *a, const void *b)
{
    const mt_rank *x = (const mt_rank *)a;
    const mt_rank *y = (const mt_rank *)b;
    if (before(x, y)) return -1;
    if (before(y, x)) return 1;
    return 0;
}

int orc_topk_mt(const float *g, float *e, int64_t d, float lr, int64_t k,
                int32_t *idx, float *val)
{
    if (k > d) k = d;
    if (k < 0) k = 0;
    const int nc = omp_get_max_threads();
    mt_rank *rank = (mt_rank *)malloc((size_t)(d > 0 ? d : 1) * sizeof *rank);
    unsigned char *sel = (unsigned char *)calloc((size_t)(d > 0 ? d : 1), 1);
    int64_t *head = (int64_t *)calloc((size_t)nc + 1, sizeof *head);
    int64_t *out = (int64_t *)calloc((size_t)nc + 1, sizeof *out);
    if (!rank || !sel || !head || !out) {
        free(rank);
        free(sel);
        free(head);
        free(out);
        return -1;
    }
    /* p into e, and each chunk's coordinates in the Top-k order */
#pragma omp parallel for schedule(static, 1) num_threads(nc)
    for (int c = 0; c < nc; c++) {
        int64_t lo, hi;
        chunk_bounds(d, nc, c, &lo, &hi);
        for (int64_t i = lo; i < hi; i++) {
            e[i] = ef_accumulate(e[i], lr, g[i]);
            rank[i].key = magnitude_key(e[i]);
            rank[i].index = (int32_t)i;
        }
        qsort(rank + lo, (size_t)(hi - lo), sizeof *rank, rank_cmp);
    }
    /* the first k of the whole order: repeatedly the best chunk head */
    for (int c = 0; c < nc; c++) {
        int64_t lo, hi;
        chunk_bounds(d, nc, c, &lo, &hi);
        head[c] = lo;
    }
    for (int64_t j = 0; j < k; j++) {
        int best = -1;
        for (int c = 0; c < nc; c++) {
            int64_t lo, hi;
            chunk_bounds(d, nc, c, &lo, &hi);
            if (head[c] >= hi) continue;
            if (best < 0 || before(&rank[head[c]], &rank[head[best]])) best = c;
        }
        sel[rank[head[best]].index] = 1;
        head[best]++;
    }
    /* the kept pairs in ascending index order; e_{t+1} */
#pragma omp parallel for schedule(static, 1) num_threads(nc)
    for (int c = 0; c < nc; c++) {
        int64_t lo, hi, n = 0;
        chunk_bounds(d, nc, c, &lo, &hi);
        for (int64_t i = lo; i < hi; i++) n += sel[i];
        out[c + 1] = n;
    }
    for (int c = 0; c < nc; c++) out[c + 1] += out[c];
#pragma omp parallel for schedule(static, 1) num_threads(nc)
    for (int c = 0; c < nc; c++) {
        int64_t lo, hi;
        chunk_bounds(d, nc, c, &lo, &hi);
        int64_t o = out[c];
        for (int64_t i = lo; i < hi; i++) {
            if (sel[i]) {
                idx[o] = (int32_t)i;
                val[o] = e[i];
                o++;
                e[i] = 0.0f;
            }
        }
    }
    free(rank);
    free(sel);
    free(head);
    free(out);
    return 0;
}

int64_t orc_topk_segmented_mt(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                              const int64_t *off, const int64_t *k, int32_t *idx, float *val)
{
    if (nseg < 1 || off[0] != 0 || off[nseg] != d) return -1;
    for (int32_t s = 0; s < nseg; s++)
        if (off[s + 1] < off[s] || k[s] < 0) return -1;
    int64_t *kout = (int64_t *)calloc((size_t)nseg + 1, sizeof *kout);
    if (!kout) return -1;
    for (int32_t s = 0; s < nseg; s++) {
        const int64_t size = off[s + 1] - off[s];
        kout[s + 1] = kout[s] + (k[s] < size ? k[s] : size);
    }
    int failed = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : failed)
    for (int32_t s = 0; s < nseg; s++) {
        const int64_t ks = kout[s + 1] - kout[s];
        if (orc_topk(g + off[s], e + off[s], off[s + 1] - off[s], lr, ks, idx + kout[s],
                     val + kout[s]) != 0) {
            failed = 1;
            continue;
        }
        for (int64_t j = 0; j < ks; j++) idx[kout[s] + j] += (int32_t)off[s];
    }
    const int64_t total = kout[nseg];
    free(kout);
    return failed ? -1 : total;
}

int orc_accumulate_mt(const int32_t *const *idx, const float *const *val,
                      const int64_t *counts, int32_t n, int64_t d, float *out)
{
    for (int32_t w = 0; w < n; w++)
        for (int64_t j = 0; j < counts[w]; j++)
            if (idx[w][j] < 0 || (int64_t)idx[w][j] >= d) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < d; i++) out[i] = 0.0f;
    for (int32_t w = 0; w < n; w++)
        for (int64_t j = 0; j < counts[w]; j++) {
            const int64_t i = idx[w][j];
            out[i] = out[i] + val[w][j];
        }
    const float fn = (float)n;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < d; i++) out[i] = out[i] / fn;
    return 0;
}
