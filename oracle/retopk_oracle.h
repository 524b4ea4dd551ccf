/*
 * retopk_oracle.h -- plain CPU oracle for the ReTopK decode step.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, obviously correct
 * statement of what the ReTopK selector and aggregator compute (Sec. 3.2-3.4,
 * Eq. 1 and Eq. 4-13 of "Recall Before You Rank: Similarity-Guided Top-K Reuse
 * for Efficient Long-Context Attention").  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it.  It shares no code, header
 * or constant table with the GPU library, and the GPU library never calls it.
 *
 * Arithmetic: inputs are float32 arrays (bf16 inputs are passed widened to
 * float32, which is exact).  Every dot product, norm, exponential and sum is
 * carried out in float64.  The only values rounded to float32 are the ones the
 * method ranks and stores: the scaled QK score fl32(fl32(q.k) * fl32(1/sqrt d)),
 * the stored normalised query fl32(q / ||q||) and the attention output.
 *
 * Conventions (indices are 0-based; "len" is the number of valid KV rows):
 *   q     [B, Hq, d]              current query of each (sequence, query head)
 *   k, v  [B, Hkv, max_len, d]    complete KV cache; row i of KV head g
 *   query head h reads KV head g = h / (Hq / Hkv)
 *   out   [B, Hq, d]              float32 attention output
 *   sel   [B, Hq, K]              selected support, ascending, padded with -1
 */
#ifndef RETOPK_ORACLE_H
#define RETOPK_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t batch;        /* B                                            */
    int32_t n_q_heads;    /* Hq                                           */
    int32_t n_kv_heads;   /* Hkv, Hq % Hkv == 0                           */
    int32_t head_dim;     /* d                                            */
    int64_t max_len;      /* rows allocated per (b, kv head) in k and v   */
    int32_t k;            /* K, support size                              */
    int32_t cache_cap;    /* C in the paper: query-support cache capacity */
    int32_t r;            /* R in the paper: retrieved entries per step   */
    int32_t window;       /* W: recent window                             */
    float   tau;          /* similarity fallback threshold                */
    int32_t refresh;      /* T_r in the paper: refresh period, 0 = off    */
    int32_t retrieval;    /* 0: the R most similar entries (Eq. 7); 1: the R
                             most recently inserted ones, the recent-R
                             alternative of the component ablation (Table 3) */
} orc_config;

/* Path codes, one per (b, query head) and step. */
enum { ORC_REUSE = 0, ORC_FALLBACK = 1, ORC_REFRESH = 2, ORC_COLD = 3 };

/* Optional per-step diagnostics; every pointer may be NULL. */
typedef struct {
    int8_t  *path;       /* [B*Hq]                                        */
    double  *rho_max;    /* [B*Hq]  NaN when not computed                 */
    int32_t *retrieved;  /* [B*Hq*r] slot ids, best first, -1 padded      */
    int32_t *n_cand;     /* [B*Hq]  |candidate set| on reuse, else 0      */
    int32_t *cand;       /* [B*Hq*(r*K+W)] ascending, -1 padded           */
    float   *sel_score;  /* [B*Hq*K] score of each sel entry, NaN padded  */
} orc_info;

typedef struct orc_handle orc_handle;

/* Status: 0 = ok, -1 = bad argument, -3 = out of memory. */
int  orc_create(const orc_config *cfg, orc_handle **out);
void orc_destroy(orc_handle *h);

/* Prompt-tail initialisation of the query-support cache (Sec. 3.3).
 * q_tail [B, Hq, n, d] holds the queries at positions prefill_len-n .. prefill_len-1;
 * query u gets its Exact Top-K support over the causal prefix len = prefill_len-n+u+1
 * and is inserted.  head_mask [B*Hq] (nullable) restricts the work to some heads. */
int orc_prefill_init(orc_handle *h, const float *q_tail, int32_t n, const float *k,
                     const float *v, int64_t prefill_len, const uint8_t *head_mask);

/* One ReTopK decode step over all (b, h) at KV length len (Eq. 5-13). */
int orc_decode_step(orc_handle *h, const float *q, const float *k, const float *v,
                    int64_t len, float *out, int32_t *sel, orc_info *info,
                    const uint8_t *head_mask);

/* Stateless Exact Top-K attention (Eq. 1, Eq. 4, Eq. 12). */
int orc_exact(const orc_config *cfg, const float *q, const float *k, const float *v,
              int64_t len, float *out, int32_t *sel, float *sel_score,
              const uint8_t *head_mask);

/* Cache state, copied out / in (host arrays):
 * qbar [B*Hq, C, d] float, supp [B*Hq, C, K] int32, cnt [B*Hq, C] int32. */
int orc_get_state(const orc_handle *h, float *qbar, int32_t *supp, int32_t *cnt,
                  int64_t *n_inserted, int64_t *t_dec);
int orc_set_state(orc_handle *h, const float *qbar, const int32_t *supp, const int32_t *cnt,
                  int64_t n_inserted, int64_t t_dec);

/* Helpers for the test suite: the ranked score of rows idx[0..n) of krows
 * against q, and the normalised query. */
void orc_scores(const float *q, const float *krows, int32_t d, int64_t n,
                const int32_t *idx, float *out);
void orc_normalize(const float *q, int32_t d, float *qbar);

/* Eq. 10 then Eq. 12 over a given index set idx[0..n): the output an attention
 * step produces when its support is exactly that set (used to check an output
 * computed on an equally valid near-tie support). */
void orc_attend(const float *q, const float *krows, const float *vrows, int32_t d, int64_t n,
                const int32_t *idx, float *out);

#ifdef __cplusplus
}
#endif
#endif
