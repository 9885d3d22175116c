/* The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer,
 * run over edge cases (empty vectors, k = 0 and k = d, a zero capacity,
 * bad layouts and indices, special values).  Prints "ok" and exits 0 when
 * every return value is the expected one and no sanitizer reported. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void orc_ht(const float *g, float *e, int64_t d, float lr, float lambda, int32_t *idx,
            float *val, int64_t cap, int64_t *count);
int orc_topk(const float *g, float *e, int64_t d, float lr, int64_t k, int32_t *idx, float *val);
int64_t orc_topk_segmented(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                           const int64_t *off, const int64_t *k, int32_t *idx, float *val);
int orc_accumulate(const int32_t *const *idx, const float *const *val, const int64_t *counts,
                   int32_t n, int64_t d, float *out);
int orc_update(const int32_t *const *idx, const float *const *val, const int64_t *counts,
               int32_t n, int64_t d, int mode, float *x, float *m, float beta, float gamma);

static int failures = 0;
#define EXPECT(c) do { if (!(c)) { printf("FAIL line %d: %s\n", __LINE__, #c); failures++; } } while (0)

int main(void)
{
    enum { D = 4099 };
    float *g = malloc(D * sizeof *g), *e = malloc(D * sizeof *e), *val = malloc(D * sizeof *val);
    int32_t *idx = malloc(D * sizeof *idx);
    uint32_t s = 12345u;
    for (int i = 0; i < D; i++) {
        s = s * 1664525u + 1013904223u;
        g[i] = ((float)(s >> 8) / 16777216.0f - 0.5f) * 1e-3f;
        e[i] = 0.0f;
    }
    g[0] = NAN; g[1] = INFINITY; g[2] = -INFINITY; g[3] = -0.0f; g[4] = 1e-45f;
    int64_t count = -1;
    orc_ht(g, e, 0, 0.1f, 1e-5f, idx, val, 0, &count);
    EXPECT(count == 0);
    orc_ht(g, e, D, 0.1f, 2e-5f, idx, val, 0, &count);         /* nothing written, true count */
    EXPECT(count > 0);
    orc_ht(g, e, D, 0.1f, 0.0f, idx, val, D, &count);
    EXPECT(count == D - 1);                                      /* NaN is never kept */
    for (int64_t k = 0; k <= D; k += D / 3 + 1) EXPECT(orc_topk(g, e, D, 0.1f, k, idx, val) == 0);
    EXPECT(orc_topk(g, e, D, 0.1f, D, idx, val) == 0);
    EXPECT(orc_topk(g, e, 0, 0.1f, 0, idx, val) == 0);
    int64_t off[4] = {0, 1, 1, D}, ks[3] = {1, 5, 100};
    EXPECT(orc_topk_segmented(g, e, D, 0.1f, 3, off, ks, idx, val) == 101);
    int64_t bad[4] = {0, 7, 3, D};
    EXPECT(orc_topk_segmented(g, e, D, 0.1f, 3, bad, ks, idx, val) == -1);
    int32_t pi[3] = {0, 5, D - 1}, pj[2] = {5, D};
    float pv[3] = {1.0f, 2.0f, 3.0f};
    const int32_t *pidx[2] = {pi, pj};
    const float *pval[2] = {pv, pv};
    int64_t cnt[2] = {3, 1};
    float *out = malloc(D * sizeof *out), *m = calloc(D, sizeof *m);
    EXPECT(orc_accumulate(pidx, pval, cnt, 2, D, out) == 0);
    cnt[1] = 2;                                                  /* index D is out of range */
    EXPECT(orc_accumulate(pidx, pval, cnt, 2, D, out) == -1);
    cnt[1] = 1;
    EXPECT(orc_update(pidx, pval, cnt, 2, D, 2, out, m, 0.9f, 0.1f) == 0);
    EXPECT(orc_update(pidx, pval, cnt, 2, D, 3, out, m, 0.9f, 0.1f) == -1);
    free(g); free(e); free(val); free(idx); free(out); free(m);
    printf(failures ? "%d failures\n" : "ok\n", failures);
    return failures ? 1 : 0;
}
