/*
 * retopk.h -- C ABI of the MI355X (gfx950) ReTopK decode-step library.
 *
 * ReTopK ("Recall Before You Rank: Similarity-Guided Top-K Reuse for Efficient
 * Long-Context Attention") replaces the full-history Exact Top-K selection of
 * sparse decode attention (Eq. 1, Eq. 4) by a recall-before-rerank step
 * (Sec. 3.3): the current query is matched against a bounded per-head cache of
 * normalised past queries (Eq. 5, Eq. 6), the supports of the R most similar
 * entries are united with a recent window (Eq. 7-9), only that candidate set is
 * scored with the current query (Eq. 10) and reranked to K entries (Eq. 11), and
 * Softmax-V runs over those K rows (Eq. 12).  When the best similarity is below
 * tau, or every T_r decode steps, the step falls back to Exact Top-K instead
 * (Eq. 13, Sec. 3.4).  Either way (q_bar, support) is inserted into the cache.
 *
 * Tensor layouts (all row-major, device memory unless stated):
 *   q        [B, Hq, d]            current queries, element type = config dtype
 *   q_tail   [B, Hq, n, d]         prompt-tail queries for retopk_prefill_init
 *   k, v     [B, Hkv, max_len, d]  complete KV cache; rows [0, len) are valid
 *   out      [B, Hq, d]            float32 attention output
 *   sel      [B, Hq, K]            int32 selected support, ascending, -1 padded
 * Query head h uses KV head h / (Hq / Hkv).  The caller owns every pointer it
 * passes; the library owns the per-head caches and all workspaces, allocated in
 * retopk_create and released in retopk_destroy.  No step call allocates memory.
 *
 * Streams: the step calls are asynchronous on the HIP stream passed in
 * (a hipStream_t, NULL = the null stream); path decisions stay on the device.
 * A call on another stream than the handle's previous call first makes that
 * stream wait (on the device, through an event) for the work the previous call
 * queued, since all calls of a handle share its caches and workspaces.
 * retopk_stats, retopk_get_state, retopk_set_state and retopk_profile_read
 * synchronise the stream of the last step call.  A handle is not thread-safe:
 * calls on one handle must not overlap on the host.
 *
 * Errors: arguments are checked on the host before any device work; a failing
 * check returns RETOPK_ERR_ARG (or RETOPK_ERR_UNSUPPORTED for a shape the
 * kernels are not built for) and changes nothing.  A HIP failure returns
 * RETOPK_ERR_HIP and marks the handle broken: later step calls return
 * RETOPK_ERR_STATE.
 */
#ifndef RETOPK_H
#define RETOPK_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct retopk_handle_s *retopk_handle;

typedef enum { RETOPK_F32 = 0, RETOPK_BF16 = 1 } retopk_dtype;

typedef enum {
    RETOPK_OK = 0,
    RETOPK_ERR_ARG = -1,          /* invalid argument or null pointer          */
    RETOPK_ERR_UNSUPPORTED = -2,  /* valid, but no kernel for this shape        */
    RETOPK_ERR_OOM = -3,          /* device allocation failed in retopk_create  */
    RETOPK_ERR_HIP = -4,          /* a HIP runtime call failed                  */
    RETOPK_ERR_STATE = -5,        /* call out of order (see each function)      */
    RETOPK_ERR_TOO_LARGE = -6     /* the call needs more workspace than the     */
                                  /* fixed scratch of exact_topk_attention_noalloc */
} retopk_status;

/* Path taken by one (sequence, query head) in one step (Eq. 13). */
typedef enum {
    RETOPK_REUSE = 0,     /* recall-before-rerank (Sec. 3.3)                    */
    RETOPK_FALLBACK = 1,  /* rho_max < tau: Exact Top-K (Sec. 3.4)              */
    RETOPK_REFRESH = 2,   /* scheduled refresh, t_dec in {T_r, 2T_r, ...}       */
    RETOPK_COLD = 3       /* the cache is empty (capacity 0 or nothing inserted)*/
} retopk_path;

typedef struct {
    int32_t batch;       /* B >= 1                                               */
    int32_t n_q_heads;   /* Hq >= 1                                              */
    int32_t n_kv_heads;  /* Hkv >= 1, Hq % Hkv == 0, 1 <= Hq / Hkv <= 8           */
    int32_t head_dim;    /* d in {64, 128}                                       */
    int64_t max_len;     /* rows allocated per (b, KV head) in k and v, 1 ..     */
                         /* 2^24 (RETOPK_ERR_ARG from 2^31, else                */
                         /* RETOPK_ERR_UNSUPPORTED above 2^24)                  */
    int32_t k;           /* K: support size, 1 <= K <= 2048                      */
    int32_t cache_cap;   /* C (paper), M: cache entries per query head, 0..4096  */
    int32_t r;           /* R (paper): retrieved entries per step, 1..32         */
    int32_t window;      /* W: recent window, >= 0                               */
    float   tau;         /* fallback threshold on rho_max, finite                */
    int32_t refresh;     /* T_r (paper), P: refresh period in steps, 0 = off     */
    int32_t dtype;       /* retopk_dtype of q, k and v                           */
    int32_t retrieval;   /* 0: the R most similar cached queries (Eq. 7); 1: the  */
                         /* R most recently inserted entries (the recent-R      */
                         /* alternative of the component ablation, Table 3),    */
                         /* whose best similarity is then rho_max (Eq. 13)      */
} retopk_config;

/* Cumulative counters since retopk_create (or the last retopk_set_state). */
typedef struct {
    uint64_t steps;           /* retopk_decode_step calls                        */
    uint64_t head_steps;      /* steps x B x Hq                                  */
    uint64_t reuse;           /* head-steps per path                             */
    uint64_t fallback;
    uint64_t refresh;
    uint64_t cold;
    uint64_t kv_group_scans;  /* (b, KV head) full-history scans run             */
    uint64_t cand_sum;        /* sum of |candidate set| over reuse head-steps    */
    uint64_t cand_max;        /* largest |candidate set|                         */
} retopk_stats_t;

/* Optional per-step diagnostics of retopk_decode_step (device pointers, each may
 * be NULL).  Slots are cache positions: the i-th insertion goes to slot i mod C. */
typedef struct {
    int8_t  *path;       /* [B*Hq] retopk_path                                  */
    double  *rho_max;    /* [B*Hq] best cosine similarity; NaN when not computed */
    int32_t *retrieved;  /* [B*Hq*r] retrieved slots, best first, -1 padded     */
    int32_t *n_cand;     /* [B*Hq] |candidate set| on reuse, else 0             */
    int32_t *cand;       /* [B*Hq*(r*K+W)] candidate set ascending, -1 padded   */
} retopk_debug;

/* Create a handle: validates cfg and allocates the caches (C entries of d floats
 * and K indices per query head, Eq. 5, metadata cost of Sec. 3.5) and the step
 * workspaces on the current HIP device.  The cache starts empty.  It takes no
 * stream on purpose: it allocates and clears its memory synchronously and
 * returns only once the device has finished, so it is ordered before every later
 * call of the handle on any stream. */
retopk_status retopk_create(const retopk_config *cfg, retopk_handle *out);

/* Release everything retopk_create allocated: the per-head caches and the
 * preallocated step workspaces of Sec. 3.5.  Waits for the device first.  NULL is
 * accepted. */
retopk_status retopk_destroy(retopk_handle h);

/* Cache initialisation from the prompt tail (Sec. 3.3): q_tail holds the queries
 * at positions prefill_len-n .. prefill_len-1; query u is given its Exact Top-K
 * support over its causal prefix (len = prefill_len-n+u+1) and inserted, in
 * order.  Requires n >= 0 and n <= prefill_len <= max_len.  Does not advance the
 * decode-step counter.  Queries whose slot a later one overwrites (n > C) only
 * advance the insertion count.  bf16 handles score many positions of every head
 * per launch on the matrix cores (kernel id 7) with up to 2 GiB of temporary
 * device memory, and return after the stream has finished that work; when the
 * memory is not available, and for f32, the queries run one position at a time
 * through the decode step's exact path, asynchronously. */
retopk_status retopk_prefill_init(retopk_handle h, const void *q_tail, int32_t n,
                                  const void *k, const void *v, int64_t prefill_len,
                                  void *stream);

/* One ReTopK decode step for every (sequence, query head) over KV rows [0, len)
 * (Sec. 3.3-3.4).  The path is chosen per head on the device by Eq. 13, with
 * t_dec = number of earlier decode steps (the first step is t_dec = 0).  Writes
 * out (float32) and, when non-NULL, sel and the dbg arrays; inserts (q_bar,
 * support) into every head's cache.  len must satisfy 1 <= len <= max_len and
 * must not decrease between calls (RETOPK_ERR_STATE otherwise).  q, k and v must
 * be finite: a non-finite value leaves the outputs of the heads it reaches
 * unspecified (no memory outside the handle's buffers and the arguments is
 * touched). */
retopk_status retopk_decode_step(retopk_handle h, const void *q, const void *k, const void *v,
                                 int64_t len, float *out, int32_t *sel,
                                 const retopk_debug *dbg, void *stream);

/* Full (dense) attention for every head over rows [0, len): softmax of the scaled
 * scores of Eq. 4 over all rows, then the weighted sum of the value rows; the
 * no-selection reference of the paper's comparisons.  Same argument rules as
 * exact_topk_attention (device pointers, 16-byte aligned, 1 <= len <= max_len);
 * writes out (float32 [B, Hq, d]) only.  Two kernels: per-chunk partial results
 * in the handle's workspace, then their merge. */
retopk_status full_attention(retopk_handle h, const void *q, const void *k, const void *v,
                             int64_t len, float *out, void *stream);

/* Measurement aid (no part of the method): reads `bytes` of device memory at `src`
 * once with a plain streaming kernel, the practical HBM read ceiling that the
 * benchmark reports beside the published peak.  src must be 16-byte aligned and
 * bytes a multiple of 16; *sink (device, 4 bytes) is written only if the data
 * XOR to a value no real buffer of this size is expected to give, so that the
 * reads are kept.  Asynchronous on `stream`. */
retopk_status retopk_stream_read(const void *src, int64_t bytes, uint32_t *sink, void *stream);

/* Exact Top-K attention (Eq. 1 with Eq. 4, then Eq. 12) for every head over rows
 * [0, len): the full-history baseline.  Uses the handle's workspaces only; the
 * caches and counters are untouched. */
retopk_status exact_topk_attention(retopk_handle h, const void *q, const void *k,
                                   const void *v, int64_t len, float *out, int32_t *sel,
                                   void *stream);

/* Size of the fixed device scratch array behind exact_topk_attention_noalloc,
 * in MiB (one copy per GPU the library runs on, held until the process ends). */
#define RETOPK_NOALLOC_SCRATCH_MB 64

/* exact_topk_attention for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  No handle: cfg describes the layer as for retopk_create (only
 * its shape fields, K and dtype matter here) and is validated the same way; q,
 * k, v, len, out, sel and stream are as for exact_topk_attention, and the
 * result is the same (the same kernels run).  The workspaces come from a fixed
 * array of RETOPK_NOALLOC_SCRATCH_MB MiB of device memory inside the library,
 * of which one call uses, with BH = batch * n_q_heads and
 * R = 4096 * ceil(len / 4096),
 *   BH * (12 * R + 8192 + 4 * R / 4096 + 32) bytes (each of the five parts
 *   rounded up to 256 bytes);
 * a larger call returns RETOPK_ERR_TOO_LARGE before any device work (the 128K
 * layer of 32 query heads, len 131 328, needs 52 MB).  Nothing is allocated:
 * neither hipMalloc nor hipFree nor any allocating library routine is called
 * (the first call on a device looks up the array's address there).  Every call
 * on one GPU shares that GPU's array: calls that overlap on one GPU (different
 * streams or host threads without ordering between them) race and give
 * undefined results.  Each call clears what must start at zero with a kernel
 * (no memset node), so it can be captured in a HIP graph. */
retopk_status exact_topk_attention_noalloc(const retopk_config *cfg, const void *q,
                                           const void *k, const void *v, int64_t len,
                                           float *out, int32_t *sel, void *stream);

/* Read the cumulative counters (synchronises): head-steps per path of Eq. 13 --
 * the path mix of Sec. 4.2 (reuse / fallback / refresh shares), the reuse share
 * of Table 2 and the exact-path share of the component ablation (Table 3) -- the
 * full-history scans the exact path ran, and the candidate-set sizes, bounded by
 * Eq. 14. */
retopk_status retopk_stats(retopk_handle h, retopk_stats_t *out);

/* Copy the cache state to host arrays (synchronises):
 * qbar [B*Hq, C, d] float, supp [B*Hq, C, K] int32 (-1 padded), cnt [B*Hq, C];
 * n_inserted = insertions so far, t_dec = decode steps so far.  Any pointer may
 * be NULL. */
retopk_status retopk_get_state(retopk_handle h, float *qbar, int32_t *supp, int32_t *cnt,
                               int64_t *n_inserted, int64_t *t_dec);

/* Replace the cache state from host arrays laid out as in retopk_get_state
 * (synchronous).  Resets the counters and the len monotonicity check. */
retopk_status retopk_set_state(retopk_handle h, const float *qbar, const int32_t *supp,
                               const int32_t *cnt, int64_t n_inserted, int64_t t_dec);

/* Per-kernel timing with HIP events attached to each kernel's dispatch, on the
 * launch stream.  retopk_profile(h, 1) clears and starts recording,
 * retopk_profile(h, 0) stops.  retopk_profile_read (synchronises) fills, for
 * kernel ids 0 .. n_kernels-1, the number of launches and their summed duration
 * in milliseconds; it returns RETOPK_ERR_STATE if more launches were recorded
 * than the event pool holds (65536).  Kernel ids, in the order of a step:
 *   0 retopk_sim     query-cache similarities and Top-R (decode steps that select)
 *   1 retopk_score   candidate gathering and scoring plus the full-history scans
 *                    of fallback heads (decode steps that select)
 *   2 retopk_scan    the scoring kernel when every head scans its full history
 *                    (refresh, cold, Exact Top-K, prefill)
 *   3 retopk_filter  threshold bucket and survivor compaction
 *   4 retopk_final   exact Top-K, Softmax-V, cache insert
 *   5 dense_chunk    full_attention: per-chunk softmax and value sums
 *   6 dense_merge    full_attention: merge of the chunks
 *   7 prefill_score  bf16 prefill: scores of many prompt-tail positions of every
 *                    head (matrix cores); retopk_filter and retopk_final select */
retopk_status retopk_profile(retopk_handle h, int32_t enable);
retopk_status retopk_profile_read(retopk_handle h, int32_t n_kernels, uint64_t *launches,
                                  double *total_ms);
const char *retopk_kernel_name(int32_t kernel_id);   /* NULL past the last id */

const char *retopk_status_string(retopk_status s);

#ifdef __cplusplus
}
#endif
#endif
