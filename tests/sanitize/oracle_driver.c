/* The CPU oracle on randomised small problems, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer: random shapes, page sizes,
 * block tables and visible-key counts, one and several threads (the results
 * must be bit-identical), softmax weights requested or not, partial results
 * merged back into the whole, and arguments the oracle must refuse.  Prints
 * "ok" when every check holds. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int32_t mwo_paged_attention(int32_t n_rows, int32_t hq, int32_t hkv, int32_t d, int32_t s, double scale,
                            const uint16_t *q, const uint16_t *k_pool, const uint16_t *v_pool, int32_t num_pages,
                            const int32_t *block_tables, int32_t bt_stride, const int32_t *row_table,
                            const int32_t *row_nvis, double *out, double *probs, int32_t probs_stride,
                            int32_t n_threads);
int32_t mwo_merge_parts(int32_t n_parts, int32_t d, const double *m, const double *l, const double *o, double *out);
int32_t mwo_partial(int32_t hq, int32_t hkv, int32_t d, int32_t s, double scale, const uint16_t *q_row,
                    const uint16_t *k_pool, const uint16_t *v_pool, int32_t num_pages, const int32_t *bt, int32_t h,
                    int32_t j0, int32_t j1, double *m_out, double *l_out, double *o_out);

static uint64_t g_state = 0x2545F4914F6CDD1Dull;
static uint32_t next_u32(void) {
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return (uint32_t)((g_state * 0x9E3779B97F4A7C15ull) >> 32);
}
static int uniform(int lo, int hi) { return lo + (int)(next_u32() % (uint32_t)(hi - lo + 1)); }
/* a bf16 pattern of a value in about [-4, 4) */
static uint16_t rand_bf16(void) { return (uint16_t)(((next_u32() & 1u) << 15) | (uniform(0x3C00, 0x4080) & 0x7FFF)); }

static int g_fail = 0;
static void check(int ok, const char *what, int it) {
    if (!ok) {
        fprintf(stderr, "check failed at iteration %d: %s\n", it, what);
        ++g_fail;
    }
}

int main(void) {
    const int hkvs[3] = {1, 2, 4}, ds[2] = {16, 128}, ss[3] = {1, 4, 16};
    for (int it = 0; it < 1000; ++it) {
        const int hkv = hkvs[uniform(0, 2)], hq = hkv * uniform(1, 4), d = ds[uniform(0, 1)], s = ss[uniform(0, 2)];
        const int n_tables = uniform(1, 4), stride = uniform(1, 12), num_pages = n_tables * stride + uniform(0, 5);
        const int n_rows = uniform(1, 6);
        const size_t pool_elems = (size_t)num_pages * hkv * s * d;
        uint16_t *k = malloc(pool_elems * 2), *v = malloc(pool_elems * 2), *q = malloc((size_t)n_rows * hq * d * 2);
        int32_t *bt = malloc(sizeof(int32_t) * n_tables * stride), *rt = malloc(sizeof(int32_t) * n_rows);
        int32_t *nvis = malloc(sizeof(int32_t) * n_rows);
        double *o1 = malloc(sizeof(double) * n_rows * hq * d), *o3 = malloc(sizeof(double) * n_rows * hq * d);
        double *pr = malloc(sizeof(double) * n_rows * hq * stride * s);
        for (size_t i = 0; i < pool_elems; ++i) { k[i] = rand_bf16(); v[i] = rand_bf16(); }
        for (int i = 0; i < n_rows * hq * d; ++i) q[i] = rand_bf16();
        for (int i = 0; i < n_tables * stride; ++i) bt[i] = uniform(0, num_pages - 1);
        int max_nvis = 1;
        for (int r = 0; r < n_rows; ++r) {
            rt[r] = uniform(0, n_tables - 1);
            nvis[r] = uniform(1, stride * s);
            if (nvis[r] > max_nvis) max_nvis = nvis[r];
        }
        const double scale = 1.0 / sqrt((double)d);
        const int want = uniform(0, 1);
        check(mwo_paged_attention(n_rows, hq, hkv, d, s, scale, q, k, v, num_pages, bt, stride, rt, nvis, o1,
                                  want ? pr : NULL, want ? stride * s : 0, 1) == 0, "one thread", it);
        check(mwo_paged_attention(n_rows, hq, hkv, d, s, scale, q, k, v, num_pages, bt, stride, rt, nvis, o3, NULL, 0,
                                  uniform(2, 5)) == 0, "threads", it);
        check(memcmp(o1, o3, sizeof(double) * n_rows * hq * d) == 0, "bit-identical for any thread count", it);
        if (want)
            for (int r = 0; r < n_rows; ++r)
                for (int h = 0; h < hq; ++h) {
                    double sum = 0.0;
                    for (int j = 0; j < nvis[r]; ++j) sum += pr[((size_t)r * hq + h) * stride * s + j];
                    check(fabs(sum - 1.0) < 1e-12, "weights sum to one", it);
                }
        /* partials over a cut of the first row's keys, merged back */
        {
            const int r = 0, h = uniform(0, hq - 1), L = nvis[r], cut = uniform(0, L);
            double m[2], l[2], *o = malloc(sizeof(double) * 2 * d), *w = malloc(sizeof(double) * d);
            const int32_t *row = bt + (size_t)rt[r] * stride;
            check(mwo_partial(hq, hkv, d, s, scale, q, k, v, num_pages, row, h, 0, cut, &m[0], &l[0], o) == 0 &&
                  mwo_partial(hq, hkv, d, s, scale, q, k, v, num_pages, row, h, cut, L, &m[1], &l[1], o + d) == 0,
                  "partials", it);
            check(mwo_merge_parts(2, d, m, l, o, w) == 0, "merge", it);
            for (int e = 0; e < d; ++e) check(fabs(w[e] - o1[(size_t)h * d + e]) < 1e-9, "merge = whole", it);
            free(o);
            free(w);
        }
        /* arguments the oracle must refuse: a page outside the pool, hq not a multiple of hkv */
        {
            const int32_t saved = bt[0];
            bt[0] = num_pages;
            nvis[0] = 1;
            rt[0] = 0;
            check(mwo_paged_attention(1, hq, hkv, d, s, scale, q, k, v, num_pages, bt, stride, rt, nvis, o1, NULL, 0,
                                      1) != 0, "page outside the pool refused", it);
            bt[0] = saved;
            if (hkv > 1)
                check(mwo_paged_attention(1, hkv + 1, hkv, d, s, scale, q, k, v, num_pages, bt, stride, rt, nvis, o1,
                                          NULL, 0, 1) != 0, "hq not a multiple of hkv refused", it);
        }
        free(k); free(v); free(q); free(bt); free(rt); free(nvis); free(o1); free(o3); free(pr);
    }
    if (g_fail) return 1;
    printf("ok\n");
    return 0;
}
