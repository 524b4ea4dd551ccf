/*
 * retopk_oracle.c -- plain CPU oracle for the ReTopK decode step.
 *
 * TEST INFRASTRUCTURE ONLY (see retopk_oracle.h).  Single-threaded C11, no
 * intrinsics, no blocking or fusion: every function below is one step of the
 * method written the way the paper states it, with float64 arithmetic.
 *
 * Readings where the paper leaves a choice open (each one is listed, with its
 * reason, in the design notes of the repository):
 *   - indices are 0-based; the recent window of Eq. 8 is [max(0, len-W), len);
 *   - the ranked score is fl32(fl32(q.k) * fl32(1/sqrt d)); ties in Top-K are
 *     broken towards the lower index, and -0.0 ranks equal to +0.0;
 *   - ties in Top-R (Eq. 7) are broken towards the more recently inserted entry;
 *   - fallback is strict (rho_max < tau reuses at equality);
 *   - the first decode step has t_dec = 0, so refreshes happen at
 *     t_dec = T_r, 2 T_r, ... (Eq. 13) and never on the first step;
 *   - an empty cache (nothing inserted yet, or capacity 0) takes the exact path
 *     ("cold"), before the refresh test;
 *   - when fewer than K candidates (or keys) exist, all of them are selected;
 *   - supports are stored in ascending index order.
 */
#include "retopk_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

struct orc_handle {
    orc_config cfg;
    float   *qbar;   /* [B*Hq][C][d]  normalised cached queries (Eq. 5)   */
    int32_t *supp;   /* [B*Hq][C][K]  cached supports, ascending          */
    int32_t *cnt;    /* [B*Hq][C]     valid entries of each support       */
    int64_t  n_ins;  /* entries inserted so far (every head inserts once per step) */
    int64_t  t_dec;  /* decode steps taken so far                          */
};

typedef struct {
    float   s;   /* ranked score */
    int32_t i;   /* key index    */
} scored_key;

/* ------------------------------------------------------------------------ */
/* Basic definitions                                                          */
/* ------------------------------------------------------------------------ */

/* The scaled QK score of Eq. 4 / Eq. 10, q^T k / sqrt(d), as the fp32 value that
 * both implementations rank: the dot product rounded to fp32, times fl32(1/sqrt d). */
static float qk_score(const float *q, const float *krow, int d)
{
    double dot = 0.0;
    for (int j = 0; j < d; ++j)
        dot += (double)q[j] * (double)krow[j];
    float inv_sqrt_d = (float)(1.0 / sqrt((double)d));
    return (float)dot * inv_sqrt_d;
}

/* Total order used by TopK in Eq. 1 and Eq. 11: higher score first, then lower
 * index.  Comparing floats with < and > ranks -0.0 equal to +0.0. */
static int cmp_rank(const void *a, const void *b)
{
    const scored_key *x = (const scored_key *)a;
    const scored_key *y = (const scored_key *)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    if (x->i < y->i) return -1;
    if (x->i > y->i) return 1;
    return 0;
}

static int cmp_index(const void *a, const void *b)
{
    const scored_key *x = (const scored_key *)a;
    const scored_key *y = (const scored_key *)b;
    return (x->i > y->i) - (x->i < y->i);
}

static int cmp_int32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* TopK over the given (score, index) list (Eq. 1 over all keys, Eq. 11 over the
 * candidate set): sort by the ranking order and keep the first min(K, n).  The
 * kept entries are then put in ascending index order.  Returns the count kept. */
static int64_t top_k(scored_key *list, int64_t n, int32_t K)
{
    qsort(list, (size_t)n, sizeof(scored_key), cmp_rank);
    int64_t kept = n < K ? n : K;
    qsort(list, (size_t)kept, sizeof(scored_key), cmp_index);
    return kept;
}

/* Sparse Softmax-V aggregation of Eq. 12 over the selected entries. */
static void softmax_v(const scored_key *sel, int64_t n, const float *vbase, int d,
                      float *out)
{
    double m = -INFINITY;
    for (int64_t t = 0; t < n; ++t)
        if ((double)sel[t].s > m) m = (double)sel[t].s;
    double *acc = (double *)calloc((size_t)d, sizeof(double));
    double l = 0.0;
    for (int64_t t = 0; t < n; ++t) {
        double w = exp((double)sel[t].s - m);
        const float *vrow = vbase + (int64_t)sel[t].i * d;
        l += w;
        for (int j = 0; j < d; ++j)
            acc[j] += w * (double)vrow[j];
    }
    for (int j = 0; j < d; ++j)
        out[j] = n > 0 ? (float)(acc[j] / l) : 0.0f;
    free(acc);
}

/* q_bar = q / ||q||_2 of Eq. 5 and Eq. 6, stored as fp32.  A zero query maps to 0. */
void orc_normalize(const float *q, int32_t d, float *qbar)
{
    double ss = 0.0;
    for (int j = 0; j < d; ++j)
        ss += (double)q[j] * (double)q[j];
    double nrm = sqrt(ss);
    for (int j = 0; j < d; ++j)
        qbar[j] = nrm > 0.0 ? (float)((double)q[j] / nrm) : 0.0f;
}

void orc_scores(const float *q, const float *krows, int32_t d, int64_t n,
                const int32_t *idx, float *out)
{
    for (int64_t t = 0; t < n; ++t)
        out[t] = qk_score(q, krows + (int64_t)idx[t] * d, d);
}

void orc_attend(const float *q, const float *krows, const float *vrows, int32_t d, int64_t n,
                const int32_t *idx, float *out)
{
    scored_key *list = (scored_key *)malloc((size_t)(n > 0 ? n : 1) * sizeof(scored_key));
    for (int64_t t = 0; t < n; ++t) {
        list[t].s = qk_score(q, krows + (int64_t)idx[t] * d, d);
        list[t].i = idx[t];
    }
    qsort(list, (size_t)n, sizeof(scored_key), cmp_index);
    softmax_v(list, n, vrows, d, out);
    free(list);
}

/* ------------------------------------------------------------------------ */
/* Exact Top-K attention for one query head (Eq. 1, Eq. 4, Eq. 12)           */
/* ------------------------------------------------------------------------ */

/* Scores every key i < len, keeps the top min(K, len) and aggregates V over
 * them.  sel / sel_score receive K entries (padded), out receives d values.
 * Returns the support size. */
static int64_t exact_head(const float *q, const float *kbase, const float *vbase,
                          int d, int64_t len, int32_t K, float *out,
                          int32_t *sel, float *sel_score)
{
    scored_key *list = (scored_key *)malloc((size_t)(len > 0 ? len : 1) * sizeof(scored_key));
    for (int64_t i = 0; i < len; ++i) {
        list[i].s = qk_score(q, kbase + i * d, d);
        list[i].i = (int32_t)i;
    }
    int64_t kept = top_k(list, len, K);
    if (out) softmax_v(list, kept, vbase, d, out);
    for (int32_t t = 0; t < K; ++t) {
        if (sel) sel[t] = t < kept ? list[t].i : -1;
        if (sel_score) sel_score[t] = t < kept ? list[t].s : NAN;
    }
    free(list);
    return kept;
}

/* ------------------------------------------------------------------------ */
/* Handle                                                                     */
/* ------------------------------------------------------------------------ */

static int config_ok(const orc_config *c)
{
    if (!c) return 0;
    if (c->batch < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 1) return 0;
    if (c->n_q_heads % c->n_kv_heads != 0) return 0;
    if (c->max_len < 1 || c->max_len > INT32_MAX) return 0;
    if (c->k < 1 || c->cache_cap < 0 || c->r < 1 || c->window < 0 || c->refresh < 0) return 0;
    if (!isfinite(c->tau)) return 0;
    if (c->retrieval != 0 && c->retrieval != 1) return 0;
    return 1;
}

int orc_create(const orc_config *cfg, orc_handle **out)
{
    if (!out || !config_ok(cfg)) return -1;
    orc_handle *h = (orc_handle *)calloc(1, sizeof(orc_handle));
    if (!h) return -3;
    h->cfg = *cfg;
    size_t heads = (size_t)cfg->batch * cfg->n_q_heads;
    size_t C = (size_t)cfg->cache_cap;
    h->qbar = (float *)calloc(heads * C * cfg->head_dim + 1, sizeof(float));
    h->supp = (int32_t *)calloc(heads * C * cfg->k + 1, sizeof(int32_t));
    h->cnt = (int32_t *)calloc(heads * C + 1, sizeof(int32_t));
    if (!h->qbar || !h->supp || !h->cnt) {
        orc_destroy(h);
        return -3;
    }
    *out = h;
    return 0;
}

void orc_destroy(orc_handle *h)
{
    if (!h) return;
    free(h->qbar);
    free(h->supp);
    free(h->cnt);
    free(h);
}

static const float *q_row(const orc_config *c, const float *q, int b, int hq)
{
    return q + ((int64_t)b * c->n_q_heads + hq) * c->head_dim;
}

static const float *kv_base(const orc_config *c, const float *kv, int b, int hq)
{
    int group = c->n_q_heads / c->n_kv_heads;   /* query heads per KV head */
    int g = hq / group;
    return kv + ((int64_t)b * c->n_kv_heads + g) * c->max_len * c->head_dim;
}

/* FIFO insert of (q_bar, S) into the head's cache (Eq. 5; insertion after either
 * path, Sec. 3.3 and Sec. 3.4).  The slot is the insertion count modulo C, so the
 * cache always holds the last min(n, C) inserted entries. */
static void cache_insert(orc_handle *h, int64_t head, const float *qbar,
                         const int32_t *sel, int64_t kept)
{
    const orc_config *c = &h->cfg;
    if (c->cache_cap == 0) return;
    int64_t slot = h->n_ins % c->cache_cap;
    int64_t e = head * c->cache_cap + slot;
    memcpy(h->qbar + e * c->head_dim, qbar, (size_t)c->head_dim * sizeof(float));
    for (int32_t t = 0; t < c->k; ++t)
        h->supp[e * c->k + t] = t < kept ? sel[t] : -1;
    h->cnt[e] = (int32_t)kept;
}

static int64_t n_valid_of(const orc_handle *h)
{
    int64_t C = h->cfg.cache_cap;
    return h->n_ins < C ? h->n_ins : C;
}

/* ------------------------------------------------------------------------ */
/* Prefill initialisation (Sec. 3.3: cache filled from the final prompt tokens) */
/* ------------------------------------------------------------------------ */

int orc_prefill_init(orc_handle *h, const float *q_tail, int32_t n, const float *k,
                     const float *v, int64_t prefill_len, const uint8_t *head_mask)
{
    if (!h || !q_tail || !k || !v || n < 0 || prefill_len < n || prefill_len > h->cfg.max_len)
        return -1;
    const orc_config *c = &h->cfg;
    int d = c->head_dim;
    int32_t *sel = (int32_t *)malloc((size_t)c->k * sizeof(int32_t));
    float *qbar = (float *)malloc((size_t)d * sizeof(float));
    for (int32_t u = 0; u < n; ++u) {
        int64_t len = prefill_len - n + u + 1;   /* causal prefix of query u */
        for (int b = 0; b < c->batch; ++b) {
            for (int hq = 0; hq < c->n_q_heads; ++hq) {
                int64_t head = (int64_t)b * c->n_q_heads + hq;
                if (head_mask && !head_mask[head]) continue;
                const float *qu = q_tail + (head * n + u) * d;
                int64_t kept = exact_head(qu, kv_base(c, k, b, hq), kv_base(c, v, b, hq),
                                          d, len, c->k, NULL, sel, NULL);
                orc_normalize(qu, d, qbar);
                cache_insert(h, head, qbar, sel, kept);
            }
        }
        if (c->cache_cap > 0) h->n_ins++;
    }
    free(sel);
    free(qbar);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* One decode step (Sec. 3.3 and Sec. 3.4)                                    */
/* ------------------------------------------------------------------------ */

int orc_decode_step(orc_handle *h, const float *q, const float *k, const float *v,
                    int64_t len, float *out, int32_t *sel, orc_info *info,
                    const uint8_t *head_mask)
{
    if (!h || !q || !k || !v || !out || len < 1 || len > h->cfg.max_len) return -1;
    const orc_config *c = &h->cfg;
    const int d = c->head_dim;
    const int32_t K = c->k, R = c->r, C = c->cache_cap;
    const int64_t cand_cap = (int64_t)R * K + c->window;
    const int64_t n_valid = n_valid_of(h);

    /* Eq. 13: refresh at t_dec in {T_r, 2T_r, ...} when T_r > 0. */
    const int refresh = c->refresh > 0 && h->t_dec > 0 && h->t_dec % c->refresh == 0;

    float *qbar = (float *)malloc((size_t)d * sizeof(float));
    double *rho = (double *)malloc((size_t)(C > 0 ? C : 1) * sizeof(double));
    int32_t *slot_order = (int32_t *)malloc((size_t)(C > 0 ? C : 1) * sizeof(int32_t));
    int32_t *raw = (int32_t *)malloc((size_t)cand_cap * sizeof(int32_t));
    scored_key *list = (scored_key *)malloc((size_t)(len > cand_cap ? len : cand_cap) * sizeof(scored_key));
    int32_t *support = (int32_t *)malloc((size_t)K * sizeof(int32_t));

    for (int b = 0; b < c->batch; ++b) {
        for (int hq = 0; hq < c->n_q_heads; ++hq) {
            const int64_t head = (int64_t)b * c->n_q_heads + hq;
            if (head_mask && !head_mask[head]) continue;
            const float *qh = q_row(c, q, b, hq);
            const float *kb = kv_base(c, k, b, hq);
            const float *vb = kv_base(c, v, b, hq);
            float *oh = out + head * d;

            orc_normalize(qh, d, qbar);

            int path;
            double rho_max = NAN;
            if (n_valid == 0) {
                path = ORC_COLD;
            } else if (refresh) {
                path = ORC_REFRESH;
            } else {
                /* Eq. 6: cosine similarity to every cached query.  rho_max is
                 * the largest similarity among the entries retrieval will use:
                 * all of them for Eq. 7 (its best one is retrieved), the R most
                 * recent ones for recent-R retrieval. */
                rho_max = -INFINITY;
                for (int64_t s = 0; s < n_valid; ++s) {
                    const float *cq = h->qbar + (head * C + s) * d;
                    double acc = 0.0;
                    for (int j = 0; j < d; ++j)
                        acc += (double)qbar[j] * (double)cq[j];
                    rho[s] = acc;
                    const int64_t age = ((h->n_ins - 1 - s) % C + C) % C;
                    const int counted = c->retrieval == 0 || age < R;
                    if (counted && acc > rho_max) rho_max = acc;
                }
                /* Eq. 13 second case, Sec. 3.4: fall back when rho_max < tau. */
                path = rho_max < (double)c->tau ? ORC_FALLBACK : ORC_REUSE;
            }

            int64_t kept;
            int64_t n_cand = 0;
            int32_t n_ret = 0;
            if (path == ORC_REUSE) {
                /* Eq. 7: the R most similar entries; equal similarity goes to the
                 * newer insertion.  Selection sort keeps this readable. */
                for (int64_t s = 0; s < n_valid; ++s) slot_order[s] = (int32_t)s;
                n_ret = (int32_t)(n_valid < R ? n_valid : R);
                for (int32_t a = 0; a < n_ret; ++a) {
                    int64_t best = a;
                    for (int64_t s = a + 1; s < n_valid; ++s) {
                        int32_t x = slot_order[s], y = slot_order[best];
                        int64_t age_x = ((h->n_ins - 1 - x) % C + C) % C;
                        int64_t age_y = ((h->n_ins - 1 - y) % C + C) % C;
                        const int newer = age_x < age_y;
                        if (c->retrieval == 0 ? (rho[x] > rho[y] || (rho[x] == rho[y] && newer))
                                              : newer)
                            best = s;
                    }
                    int32_t tmp = slot_order[a];
                    slot_order[a] = slot_order[best];
                    slot_order[best] = tmp;
                }
                /* Eq. 8 and Eq. 9: union of the retrieved supports and the recent
                 * window, deduplicated. */
                int64_t n_raw = 0;
                for (int32_t a = 0; a < n_ret; ++a) {
                    int64_t e = head * C + slot_order[a];
                    for (int32_t t = 0; t < h->cnt[e]; ++t)
                        raw[n_raw++] = h->supp[e * K + t];
                }
                int64_t w0 = len - c->window > 0 ? len - c->window : 0;
                for (int64_t i = w0; i < len; ++i)
                    raw[n_raw++] = (int32_t)i;
                qsort(raw, (size_t)n_raw, sizeof(int32_t), cmp_int32);
                for (int64_t t = 0; t < n_raw; ++t)
                    if (n_cand == 0 || raw[t] != raw[n_cand - 1]) raw[n_cand++] = raw[t];
                /* Eq. 10 and Eq. 11: exact current-query scores on the candidates,
                 * then TopK over them. */
                for (int64_t t = 0; t < n_cand; ++t) {
                    list[t].s = qk_score(qh, kb + (int64_t)raw[t] * d, d);
                    list[t].i = raw[t];
                }
                kept = top_k(list, n_cand, K);
            } else {
                /* Exact Top-K over the full history (Eq. 1 with Eq. 4). */
                for (int64_t i = 0; i < len; ++i) {
                    list[i].s = qk_score(qh, kb + i * d, d);
                    list[i].i = (int32_t)i;
                }
                kept = top_k(list, len, K);
            }

            /* Eq. 12 on the selected support. */
            softmax_v(list, kept, vb, d, oh);
            for (int32_t t = 0; t < K; ++t)
                support[t] = t < kept ? list[t].i : -1;
            if (sel)
                memcpy(sel + head * K, support, (size_t)K * sizeof(int32_t));

            if (info) {
                if (info->path) info->path[head] = (int8_t)path;
                if (info->rho_max) info->rho_max[head] = rho_max;
                if (info->retrieved)
                    for (int32_t a = 0; a < R; ++a)
                        info->retrieved[head * R + a] = a < n_ret ? slot_order[a] : -1;
                if (info->n_cand) info->n_cand[head] = (int32_t)n_cand;
                if (info->cand)
                    for (int64_t t = 0; t < cand_cap; ++t)
                        info->cand[head * cand_cap + t] = t < n_cand ? raw[t] : -1;
                if (info->sel_score)
                    for (int32_t t = 0; t < K; ++t)
                        info->sel_score[head * K + t] = t < kept ? list[t].s : NAN;
            }

            /* Sec. 3.4, last paragraph: cache (q_bar, S_hat) after either path. */
            cache_insert(h, head, qbar, support, kept);
        }
    }
    if (C > 0) h->n_ins++;
    h->t_dec++;

    free(qbar);
    free(rho);
    free(slot_order);
    free(raw);
    free(list);
    free(support);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Stateless Exact Top-K attention                                            */
/* ------------------------------------------------------------------------ */

int orc_exact(const orc_config *cfg, const float *q, const float *k, const float *v,
              int64_t len, float *out, int32_t *sel, float *sel_score,
              const uint8_t *head_mask)
{
    if (!config_ok(cfg) || !q || !k || !v || !out || len < 1 || len > cfg->max_len)
        return -1;
    const int d = cfg->head_dim;
    for (int b = 0; b < cfg->batch; ++b) {
        for (int hq = 0; hq < cfg->n_q_heads; ++hq) {
            int64_t head = (int64_t)b * cfg->n_q_heads + hq;
            if (head_mask && !head_mask[head]) continue;
            exact_head(q_row(cfg, q, b, hq), kv_base(cfg, k, b, hq), kv_base(cfg, v, b, hq),
                       d, len, cfg->k, out + head * d, sel ? sel + head * cfg->k : NULL,
                       sel_score ? sel_score + head * cfg->k : NULL);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* State access                                                               */
/* ------------------------------------------------------------------------ */

int orc_get_state(const orc_handle *h, float *qbar, int32_t *supp, int32_t *cnt,
                  int64_t *n_inserted, int64_t *t_dec)
{
    if (!h) return -1;
    const orc_config *c = &h->cfg;
    size_t e = (size_t)c->batch * c->n_q_heads * c->cache_cap;
    if (qbar) memcpy(qbar, h->qbar, e * c->head_dim * sizeof(float));
    if (supp) memcpy(supp, h->supp, e * c->k * sizeof(int32_t));
    if (cnt) memcpy(cnt, h->cnt, e * sizeof(int32_t));
    if (n_inserted) *n_inserted = h->n_ins;
    if (t_dec) *t_dec = h->t_dec;
    return 0;
}

int orc_set_state(orc_handle *h, const float *qbar, const int32_t *supp, const int32_t *cnt,
                  int64_t n_inserted, int64_t t_dec)
{
    if (!h || !qbar || !supp || !cnt || n_inserted < 0 || t_dec < 0) return -1;
    const orc_config *c = &h->cfg;
    size_t e = (size_t)c->batch * c->n_q_heads * c->cache_cap;
    memcpy(h->qbar, qbar, e * c->head_dim * sizeof(float));
    memcpy(h->supp, supp, e * c->k * sizeof(int32_t));
    memcpy(h->cnt, cnt, e * sizeof(int32_t));
    h->n_ins = c->cache_cap > 0 ? n_inserted : 0;
    h->t_dec = t_dec;
    return 0;
}
