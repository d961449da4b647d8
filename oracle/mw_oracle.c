/*
 * mw_oracle.c - plain CPU reference for paged grouped-query attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Tests, the smoke check and the benchmark's
 * CPU-baseline leg call this code; the library's GPU path never does, and the
 * two share no code: this file has its own page indexing, its own bf16
 * widening and its own softmax.
 *
 * What it computes.  The paper gives the structure, not the formula: attention
 * reads the keys and values of every processed token from a KV cache
 * (Sec. 2.1, "Architecture of LLMs"); prefill with a cache handles n new tokens
 * against L = r + n keys and decode attends to r + 1 keys (Sec. 3.3, Table
 * "tab:theory_cost"); chunked prefill must equal unchunked prefill because
 * each chunk reads the KV of every earlier chunk (Sec. 1); both phases read
 * one paged KV pool (Sec. 3.2.1 and the PagedAttention reference in Related
 * Work).  The formula itself is textbook scaled dot-product attention
 * (Vaswani et al., cited in Sec. 2.1).  Query head h reads KV head
 * h / (Hq / Hkv) (grouped-query attention with consecutive grouping).
 *
 * For one output row with `nvis` visible keys (prefill token i over prefix r:
 * nvis = r + i + 1; decode over a context of L tokens: nvis = L) and one query
 * head h:
 *
 *     kvh = h / (Hq / Hkv)
 *     for j in [0, nvis):  page = bt[j / S], slot = j % S
 *         s_j = scale * sum_d q[h][d] * K[page][kvh][slot][d]
 *     m = max_j s_j,  p_j = exp(s_j - m),  l = sum_j p_j
 *     o[h][d] = (sum_j p_j * V[page][kvh][slot][d]) / l
 *
 * Every sum runs in ascending index order in double precision; bf16 inputs
 * widen exactly.  Work is spread over threads by (row, head) item only, so the
 * result does not depend on the thread count.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MWO_OK 0
#define MWO_ERR_ARG (-1)
#define MWO_ERR_NOMEM (-2)

static double bf16_to_double(uint16_t bits) {
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

typedef struct {
    int32_t n_rows, hq, hkv, d, s, num_pages, bt_stride;
    double scale;
    const uint16_t *q, *k_pool, *v_pool;
    const int32_t *block_tables, *row_table, *row_nvis;
    double *out;
    double *probs;          /* optional: [n_rows][hq][max_nvis] */
    int32_t probs_stride;
    int32_t n_threads;
} job_t;

typedef struct {
    const job_t *job;
    int32_t tid;
    int32_t status;
} worker_t;

/* Element (token j, kv head kvh, dim e) of a pool, found through the row's
 * block table. */
static const uint16_t *pool_row(const job_t *jb, const uint16_t *pool,
                                const int32_t *bt, int32_t j, int32_t kvh) {
    int32_t page = bt[j / jb->s];
    int32_t slot = j % jb->s;
    size_t off = (((size_t)page * jb->hkv + kvh) * jb->s + slot) * jb->d;
    return pool + off;
}

static int32_t attend_one(const job_t *jb, int32_t row, int32_t h, double *scores) {
    const int32_t group = jb->hq / jb->hkv;
    const int32_t kvh = h / group;
    const int32_t nvis = jb->row_nvis[row];
    const int32_t *bt = jb->block_tables + (size_t)jb->row_table[row] * jb->bt_stride;
    const uint16_t *q = jb->q + ((size_t)row * jb->hq + h) * jb->d;
    double *o = jb->out + ((size_t)row * jb->hq + h) * jb->d;

    for (int32_t j = 0; j < nvis; ++j) {
        const uint16_t *k = pool_row(jb, jb->k_pool, bt, j, kvh);
        double dot = 0.0;
        for (int32_t e = 0; e < jb->d; ++e)
            dot += bf16_to_double(q[e]) * bf16_to_double(k[e]);
        scores[j] = dot * jb->scale;
    }
    double m = scores[0];
    for (int32_t j = 1; j < nvis; ++j)
        if (scores[j] > m) m = scores[j];
    double l = 0.0;
    for (int32_t j = 0; j < nvis; ++j) {
        scores[j] = exp(scores[j] - m);
        l += scores[j];
    }
    for (int32_t e = 0; e < jb->d; ++e) o[e] = 0.0;
    for (int32_t j = 0; j < nvis; ++j) {
        const uint16_t *v = pool_row(jb, jb->v_pool, bt, j, kvh);
        for (int32_t e = 0; e < jb->d; ++e)
            o[e] += scores[j] * bf16_to_double(v[e]);
    }
    for (int32_t e = 0; e < jb->d; ++e) o[e] /= l;
    if (jb->probs) {
        double *p = jb->probs + ((size_t)row * jb->hq + h) * jb->probs_stride;
        for (int32_t j = 0; j < nvis; ++j) p[j] = scores[j] / l;
    }
    return MWO_OK;
}

static void *worker_main(void *arg) {
    worker_t *w = (worker_t *)arg;
    const job_t *jb = w->job;
    int32_t max_nvis = 1;
    for (int32_t r = 0; r < jb->n_rows; ++r)
        if (jb->row_nvis[r] > max_nvis) max_nvis = jb->row_nvis[r];
    double *scores = (double *)malloc(sizeof(double) * (size_t)max_nvis);
    if (!scores) {
        w->status = MWO_ERR_NOMEM;
        return NULL;
    }
    const int64_t items = (int64_t)jb->n_rows * jb->hq;
    for (int64_t it = w->tid; it < items; it += jb->n_threads)
        attend_one(jb, (int32_t)(it / jb->hq), (int32_t)(it % jb->hq), scores);
    free(scores);
    w->status = MWO_OK;
    return NULL;
}

/* Checks that every key a row will read lies on a page of the pool. */
static int32_t validate(const job_t *jb) {
    if (jb->n_rows < 0 || jb->hq <= 0 || jb->hkv <= 0 || jb->hq % jb->hkv ||
        jb->d <= 0 || jb->s <= 0 || jb->num_pages <= 0 || jb->bt_stride <= 0 ||
        jb->n_threads <= 0)
        return MWO_ERR_ARG;
    for (int32_t r = 0; r < jb->n_rows; ++r) {
        int32_t nvis = jb->row_nvis[r];
        if (nvis < 1 || nvis > jb->bt_stride * jb->s || jb->row_table[r] < 0)
            return MWO_ERR_ARG;
        const int32_t *bt = jb->block_tables + (size_t)jb->row_table[r] * jb->bt_stride;
        for (int32_t p = 0; p < (nvis + jb->s - 1) / jb->s; ++p)
            if (bt[p] < 0 || bt[p] >= jb->num_pages) return MWO_ERR_ARG;
    }
    return MWO_OK;
}

/*
 * Attention for n_rows independent rows.
 *   q            [n_rows][hq][d] bf16 bits
 *   k_pool/v_pool[num_pages][hkv][s][d] bf16 bits
 *   block_tables [*][bt_stride] int32; row r uses row row_table[r]
 *   row_nvis     [n_rows] number of visible keys (positions 0..nvis-1)
 *   out          [n_rows][hq][d] double
 *   probs        optional [n_rows][hq][probs_stride] double: p_j / l
 * Returns 0, or -1 for a bad argument (including a page index outside the
 * pool), or -2 when memory runs out.
 */
int32_t mwo_paged_attention(int32_t n_rows, int32_t hq, int32_t hkv, int32_t d,
                            int32_t s, double scale, const uint16_t *q,
                            const uint16_t *k_pool, const uint16_t *v_pool,
                            int32_t num_pages, const int32_t *block_tables,
                            int32_t bt_stride, const int32_t *row_table,
                            const int32_t *row_nvis, double *out, double *probs,
                            int32_t probs_stride, int32_t n_threads) {
    job_t jb = {n_rows, hq, hkv, d, s, num_pages, bt_stride, scale, q, k_pool,
                v_pool, block_tables, row_table, row_nvis, out, probs,
                probs_stride, n_threads};
    int32_t st = validate(&jb);
    if (st != MWO_OK) return st;
    if (probs) {
        for (int32_t r = 0; r < n_rows; ++r)
            if (row_nvis[r] > probs_stride) return MWO_ERR_ARG;
    }
    if (n_threads == 1) {
        worker_t w = {&jb, 0, MWO_OK};
        worker_main(&w);
        return w.status;
    }
    pthread_t *th = (pthread_t *)calloc((size_t)n_threads, sizeof(pthread_t));
    worker_t *ws = (worker_t *)calloc((size_t)n_threads, sizeof(worker_t));
    if (!th || !ws) {
        free(th);
        free(ws);
        return MWO_ERR_NOMEM;
    }
    int32_t started = 0;
    for (int32_t t = 0; t < n_threads; ++t) {
        ws[t].job = &jb;
        ws[t].tid = t;
        ws[t].status = MWO_OK;
        if (pthread_create(&th[t], NULL, worker_main, &ws[t]) != 0) break;
        ++started;
    }
    /* Items of threads that failed to start run on this thread. */
    for (int32_t t = started; t < n_threads; ++t) worker_main(&ws[t]);
    for (int32_t t = 0; t < started; ++t) pthread_join(th[t], NULL);
    st = MWO_OK;
    for (int32_t t = 0; t < n_threads; ++t)
        if (ws[t].status != MWO_OK) st = ws[t].status;
    free(th);
    free(ws);
    return st;
}

/*
 * Log-sum-exp merge of attention over disjoint key sets (used to pin the
 * split-and-combine identity): given per-part maxima m[i], sums l[i] and
 * unnormalised outputs o[i][d] (o = sum_j exp(s_j - m) v_j over the part),
 * writes the normalised attention output over the union.  Parts with l = 0
 * (no keys) are skipped.  Returns -1 if every part is empty.
 */
int32_t mwo_merge_parts(int32_t n_parts, int32_t d, const double *m,
                        const double *l, const double *o, double *out) {
    double mstar = -INFINITY;
    for (int32_t i = 0; i < n_parts; ++i)
        if (l[i] > 0.0 && m[i] > mstar) mstar = m[i];
    if (mstar == -INFINITY) return MWO_ERR_ARG;
    double lstar = 0.0;
    for (int32_t e = 0; e < d; ++e) out[e] = 0.0;
    for (int32_t i = 0; i < n_parts; ++i) {
        if (!(l[i] > 0.0)) continue;
        double w = exp(m[i] - mstar);
        lstar += w * l[i];
        for (int32_t e = 0; e < d; ++e) out[e] += w * o[(size_t)i * d + e];
    }
    for (int32_t e = 0; e < d; ++e) out[e] /= lstar;
    return MWO_OK;
}

/*
 * Partial attention of one (row, head) over keys [j0, j1) only, in the form
 * the merge takes: m = max s_j, l = sum exp(s_j - m), o = sum exp(s_j - m) v_j.
 * An empty range gives m = -inf, l = 0, o = 0.
 */
int32_t mwo_partial(int32_t hq, int32_t hkv, int32_t d, int32_t s, double scale,
                    const uint16_t *q_row, const uint16_t *k_pool,
                    const uint16_t *v_pool, int32_t num_pages, const int32_t *bt,
                    int32_t h, int32_t j0, int32_t j1, double *m_out,
                    double *l_out, double *o_out) {
    if (hq <= 0 || hkv <= 0 || hq % hkv || h < 0 || h >= hq || j0 < 0 || j1 < j0)
        return MWO_ERR_ARG;
    job_t jb = {0, hq, hkv, d, s, num_pages, 1, scale, NULL, k_pool, v_pool,
                NULL, NULL, NULL, NULL, NULL, 0, 1};
    const int32_t kvh = h / (hq / hkv);
    const uint16_t *q = q_row + (size_t)h * d;
    for (int32_t e = 0; e < d; ++e) o_out[e] = 0.0;
    *m_out = -INFINITY;
    *l_out = 0.0;
    if (j1 == j0) return MWO_OK;
    double *sc = (double *)malloc(sizeof(double) * (size_t)(j1 - j0));
    if (!sc) return MWO_ERR_NOMEM;
    for (int32_t j = j0; j < j1; ++j) {
        if (bt[j / s] < 0 || bt[j / s] >= num_pages) {
            free(sc);
            return MWO_ERR_ARG;
        }
        const uint16_t *k = pool_row(&jb, k_pool, bt, j, kvh);
        double dot = 0.0;
        for (int32_t e = 0; e < d; ++e) dot += bf16_to_double(q[e]) * bf16_to_double(k[e]);
        sc[j - j0] = dot * scale;
    }
    double m = -INFINITY;
    for (int32_t j = 0; j < j1 - j0; ++j)
        if (sc[j] > m) m = sc[j];
    double l = 0.0;
    for (int32_t j = j0; j < j1; ++j) {
        double p = exp(sc[j - j0] - m);
        l += p;
        const uint16_t *v = pool_row(&jb, v_pool, bt, j, kvh);
        for (int32_t e = 0; e < d; ++e) o_out[e] += p * bf16_to_double(v[e]);
    }
    free(sc);
    *m_out = m;
    *l_out = l;
    return MWO_OK;
}
