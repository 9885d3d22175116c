/*
 * Plain CPU oracle for the error-feedback sparsification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the smoke check and the CPU baseline
 * leg of the benchmark do.  It shares no code, header or constant with the
 * HIP implementation.
 *
 * Paper: "Rethinking gradient sparsification as total error minimization"
 * (arXiv 2108.00951).  Every function below is the plain definition written
 * out, scalar, in ascending index order:
 *
 *   orc_ht          Algorithm 1 (the EF accumulate, compress and error-update
 *                   steps) with the hard-threshold sparsifier C_lambda,
 *                   S_lambda(x) = { i : |x[i]| >= lambda }  (section 4.2).
 *   orc_topk        the same steps with the Top-k sparsifier (section 1,
 *                   Lemma 2 in section 4.3); ties broken by lower index.
 *   orc_topk_segmented  layer-wise Top-k (Appendix C.5): orc_topk on each
 *                   segment of the vector with its own k.
 *   orc_accumulate  the exchange-and-average step of Algorithm 1,
 *                   (1/n) * sum_i Delta_i, with the sum taken in worker order.
 *   orc_update      the model update that follows it: x <- x - avg
 *                   (Algorithm 1) or the momentum form of Algorithm 2
 *                   (Appendix C.6.2).
 *
 * Arithmetic: IEEE-754 binary32, round to nearest even.  The accumulate is an
 * fp32 multiply followed by a separate fp32 add (never a fused multiply-add);
 * build with -ffp-contract=off and without fast-math (x86-64 SSE arithmetic,
 * so float expressions are evaluated in float).  No flush-to-zero.
 *
 * Readings taken where the paper is silent:
 *   - lambda is in the units of p = e + lr*g (the value that is compressed);
 *   - a kept coordinate leaves +0.0f in the error vector;
 *   - the payload holds the kept entries of p (the sparsifier copies x[i]);
 *   - Top-k emits exactly min(k, d) pairs, ranking by the bit pattern of |p|
 *     (so -0 and +0 tie), larger first, then lower index first;
 *   - the average divides the in-order fp32 sum by (float)n with one IEEE
 *     division;
 *   - AGGREGATE then DECOMPRESS in Algorithm 2 is that same average, and its
 *     step size gamma multiplies (avg + m) with m already updated.
 * Parity: pinned for all five functions (see the oracle tests).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* p_i = e_i + lr * g_i, as two separately rounded fp32 operations
 * (Algorithm 1, EF accumulate step). */
static float ef_accumulate(float e, float lr, float g)
{
    float scaled = lr * g;
    float p = e + scaled;
    return p;
}

/* Hard-threshold EF step (Algorithm 1 with C = C_lambda, section 4.2).
 *
 * g[d]      gradient, read only.
 * e[d]      error e_t on entry, e_{t+1} = p - Delta on return (in place).
 * idx, val  payload, ascending index order; at most cap pairs written.
 * *count    number of kept coordinates k_t (may exceed cap).
 */
void orc_ht(const float *g, float *e, int64_t d, float lr, float lambda,
            int32_t *idx, float *val, int64_t cap, int64_t *count)
{
    int64_t k = 0;
    for (int64_t i = 0; i < d; i++) {
        float p = ef_accumulate(e[i], lr, g[i]);
        if (fabsf(p) >= lambda) {           /* i in S_lambda(p) */
            if (k < cap) {
                idx[k] = (int32_t)i;
                val[k] = p;
            }
            k++;
            e[i] = 0.0f;                     /* p_i - p_i, written as +0 */
        } else {
            e[i] = p;                        /* p_i - 0 */
        }
    }
    *count = k;
}

/* Ranking key of a coordinate for Top-k: the bit pattern of |p|. */
typedef struct {
    uint32_t key;
    int32_t index;
} orc_rank;

static uint32_t magnitude_key(float p)
{
    uint32_t bits;
    memcpy(&bits, &p, sizeof bits);
    return bits & 0x7fffffffu;
}

/* Order: larger key first; equal keys by lower index first. */
static int rank_cmp(const void *a, const void *b)
{
    const orc_rank *x = (const orc_rank *)a;
    const orc_rank *y = (const orc_rank *)b;
    if (x->key != y->key) return x->key > y->key ? -1 : 1;
    if (x->index != y->index) return x->index < y->index ? -1 : 1;
    return 0;
}

/* Top-k EF step (Algorithm 1 with C = Top-k; Lemma 2).
 *
 * Writes exactly min(k, d) pairs in ascending index order into idx/val and
 * the new error into e (in place).  Returns 0, or -1 if scratch memory could
 * not be allocated (nothing is then written).
 */
int orc_topk(const float *g, float *e, int64_t d, float lr, int64_t k,
             int32_t *idx, float *val)
{
    if (k > d) k = d;
    if (k < 0) k = 0;
    orc_rank *rank = (orc_rank *)malloc((size_t)(d > 0 ? d : 1) * sizeof *rank);
    unsigned char *kept = (unsigned char *)calloc((size_t)(d > 0 ? d : 1), 1);
    if (!rank || !kept) {
        free(rank);
        free(kept);
        return -1;
    }
    /* p = e + lr*g, held in e for now */
    for (int64_t i = 0; i < d; i++) {
        e[i] = ef_accumulate(e[i], lr, g[i]);
        rank[i].key = magnitude_key(e[i]);
        rank[i].index = (int32_t)i;
    }
    /* Sort all coordinates by the Top-k order and keep the first k. */
    qsort(rank, (size_t)d, sizeof *rank, rank_cmp);
    for (int64_t j = 0; j < k; j++) kept[rank[j].index] = 1;
    /* Emit the kept pairs in ascending index order and form e_{t+1}. */
    int64_t out = 0;
    for (int64_t i = 0; i < d; i++) {
        if (kept[i]) {
            idx[out] = (int32_t)i;
            val[out] = e[i];
            out++;
            e[i] = 0.0f;
        }
    }
    free(rank);
    free(kept);
    return 0;
}

/* Layer-wise Top-k (Appendix C.5): the Top-k sparsifier applied to each
 * layer separately.  Segment s is coordinates [off[s], off[s+1]) and keeps
 * min(k[s], its size) of them, chosen exactly as orc_topk chooses them within
 * the segment.  The payload lists segment 0's pairs, then segment 1's, and so
 * on, each segment's in ascending index order; indices are global.  e is
 * updated in place as by orc_topk.  Returns the number of pairs written, or
 * -1 on a bad layout (off[0] != 0, off[nseg] != d, a decreasing offset, a
 * negative k) or a failed scratch allocation.
 */
int64_t orc_topk_segmented(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                           const int64_t *off, const int64_t *k, int32_t *idx, float *val)
{
    if (nseg < 1 || off[0] != 0 || off[nseg] != d) return -1;
    for (int32_t s = 0; s < nseg; s++)
        if (off[s + 1] < off[s] || k[s] < 0) return -1;
    int64_t out = 0;
    for (int32_t s = 0; s < nseg; s++) {
        const int64_t size = off[s + 1] - off[s];
        const int64_t ks = k[s] < size ? k[s] : size;
        if (orc_topk(g + off[s], e + off[s], size, lr, ks, idx + out, val + out) != 0) return -1;
        for (int64_t j = 0; j < ks; j++) idx[out + j] += (int32_t)off[s];
        out += ks;
    }
    return out;
}

/* Exchange-and-average step of Algorithm 1, one device standing in for the
 * n workers:  out = (sum over workers w = 0..n-1 of decompress(payload_w)) / n.
 *
 * Payload w holds counts[w] pairs (idx[w][j], val[w][j]); indices are
 * distinct within one payload.  Sums are formed in worker order with fp32
 * adds, then each coordinate is divided by (float)n.
 * Returns 0, or -1 when an index is outside [0, d).
 */
int orc_accumulate(const int32_t *const *idx, const float *const *val,
                   const int64_t *counts, int32_t n, int64_t d, float *out)
{
    for (int64_t i = 0; i < d; i++) out[i] = 0.0f;
    for (int32_t w = 0; w < n; w++) {
        for (int64_t j = 0; j < counts[w]; j++) {
            int64_t i = idx[w][j];
            if (i < 0 || i >= d) return -1;
            out[i] = out[i] + val[w][j];
        }
    }
    float fn = (float)n;
    for (int64_t i = 0; i < d; i++) out[i] = out[i] / fn;
    return 0;
}

/* Model update after the exchange-and-average step, applied to every
 * coordinate with the average avg of orc_accumulate:
 *   mode 1 (Algorithm 1):  x <- x - avg
 *   mode 2 (Appendix C.6.2, Algorithm 2: EF SGD with momentum and gradient
 *           compression; the paper's momentum factor is `beta` here, its
 *           learning rate `gamma`; the update uses the new m):
 *           m <- beta*m + avg ;  x <- x - gamma*(avg + m)   (new m)
 * Each operation is one separately rounded fp32 operation, in the order
 * written.  Returns 0, or -1 on an index outside [0, d) or an unknown mode.
 */
int orc_update(const int32_t *const *idx, const float *const *val,
               const int64_t *counts, int32_t n, int64_t d, int mode,
               float *x, float *m, float beta, float gamma)
{
    if (mode != 1 && mode != 2) return -1;
    float *avg = (float *)malloc((size_t)(d > 0 ? d : 1) * sizeof *avg);
    if (!avg) return -1;
    if (orc_accumulate(idx, val, counts, n, d, avg) != 0) {
        free(avg);
        return -1;
    }
    for (int64_t i = 0; i < d; i++) {
        if (mode == 1) {
            x[i] = x[i] - avg[i];
        } else {
            float decayed = beta * m[i];
            m[i] = decayed + avg[i];
            float step = avg[i] + m[i];
            float scaled = gamma * step;
            x[i] = x[i] - scaled;
        }
    }
    free(avg);
    return 0;
}
