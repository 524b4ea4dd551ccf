// retopk_api.hip -- host side of the C ABI declared in include/retopk.h:
// argument validation, device allocation, the per-step path mode, launch
// geometry and sequencing, counters, cache state access and event profiling.
#include "retopk.h"
#include "retopk_internal.h"

#include <hip/hip_ext.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

using namespace retopk;

namespace {

constexpr int kProfileMaxLaunches = 65536;
constexpr int kNumKernels = 8;
// Temporary device memory one batched prefill launch sequence may use (scores,
// survivors and histograms of U positions of every head).
constexpr size_t kPfWorkspaceBytes = (size_t)2 << 30;
// retopk_score is the scoring kernel of a decode step that selects (candidate
// blocks beside the scans of fallback heads); retopk_scan is the same kernel
// built for steps where every head takes the full-history scan.
const char *const kKernelNames[kNumKernels] = {"retopk_sim", "retopk_score", "retopk_scan",
                                               "retopk_filter", "retopk_final", "dense_chunk",
                                               "dense_merge", "prefill_score"};
enum { KID_SIM = 0, KID_SCORE = 1, KID_SCAN = 2, KID_FILTER = 3, KID_FINAL = 4, KID_DENSE = 5,
       KID_DENSE_MERGE = 6, KID_PF_SCORE = 7 };

}  // namespace

struct retopk_handle_s {
    retopk_config cfg{};
    int G = 1;
    int cand_cap = 0;
    float inv_sqrt_d = 0.0f;
    int device = 0;
    Ws w{};
    std::vector<void *> allocs;
    int64_t n_ins = 0;
    int64_t t_dec = 0;
    int64_t last_len = 0;
    bool broken = false;
    hipStream_t last_stream = nullptr;
    bool has_last = false;             // a call has queued work on last_stream
    hipEvent_t order_ev = nullptr;     // orders a call on a new stream after the last
    // host-side counters (paths decided on the host)
    uint64_t steps = 0, head_steps = 0, refresh = 0, cold = 0, host_scans = 0;
    // profiling
    bool prof = false;
    bool prof_overflow = false;
    std::vector<hipEvent_t> ev;       // 2 per launch
    std::vector<int> ev_kernel;
    size_t ev_used = 0;
};

namespace retopk {

retopk_status validate_config(const retopk_config *c)
{
    if (!c) return RETOPK_ERR_ARG;
    if (c->batch < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1) return RETOPK_ERR_ARG;
    if (c->n_q_heads % c->n_kv_heads != 0) return RETOPK_ERR_ARG;
    if (c->dtype != RETOPK_F32 && c->dtype != RETOPK_BF16) return RETOPK_ERR_ARG;
    if (c->head_dim < 1) return RETOPK_ERR_ARG;
    if (c->max_len < 1 || c->max_len >= ((int64_t)1 << 31)) return RETOPK_ERR_ARG;
    if (c->max_len > kMaxLen) return RETOPK_ERR_UNSUPPORTED;
    if (c->k < 1 || c->cache_cap < 0 || c->r < 1 || c->window < 0 || c->refresh < 0)
        return RETOPK_ERR_ARG;
    if (!std::isfinite(c->tau)) return RETOPK_ERR_ARG;
    if (c->retrieval != 0 && c->retrieval != 1) return RETOPK_ERR_ARG;
    if (c->k > kMaxK || c->cache_cap > kMaxCache || c->r > kMaxR) return RETOPK_ERR_UNSUPPORTED;
    if ((int64_t)c->batch * c->n_q_heads > kMaxHeads) return RETOPK_ERR_UNSUPPORTED;
    if ((int64_t)c->r * c->k + c->window >= ((int64_t)1 << 30)) return RETOPK_ERR_UNSUPPORTED;
    if (!shape_supported(c->dtype, c->head_dim, c->n_q_heads / c->n_kv_heads))
        return RETOPK_ERR_UNSUPPORTED;
    return RETOPK_OK;
}

StepArgs config_args(const retopk_config &c)
{
    StepArgs a{};
    a.B = c.batch;
    a.Hq = c.n_q_heads;
    a.Hkv = c.n_kv_heads;
    a.G = c.n_q_heads / c.n_kv_heads;
    a.D = c.head_dim;
    a.max_len = c.max_len;
    a.K = c.k;
    a.M = c.cache_cap;
    a.R = c.r;
    a.W = c.window;
    a.cand_cap = c.r * c.k + c.window;
    a.n_regions = (int)ceil_div(c.max_len, kFilterRows);
    a.n_dense = (int)ceil_div(c.max_len, kDenseRows);
    a.row_stride = (int64_t)a.n_regions * kFilterRows;
    a.tau = c.tau;
    a.retrieval = c.retrieval;
    a.inv_sqrt_d = (float)(1.0 / std::sqrt((double)c.head_dim));
    a.q_head_stride = c.head_dim;
    a.U = 1;
    return a;
}

// The range blocks' index ranges of a decode step that selects (Eq. 8-9 split
// over kCandRanges blocks per head).  Every row of the window [w0, len) is a
// candidate, so the window gets ranges of its own, about as many as its share
// of the candidates (W rows against R * K support entries, weighted 10 : 3),
// so that no range block gathers far more rows than the others; the ranges
// stay in index order.
void range_split(StepArgs &a)
{
    a.w0 = a.len - a.W > 0 ? a.len - a.W : 0;
    a.n_win = 0;
    if (a.W > 0) {
        const int64_t share = (10ll * kCandRanges * a.W + 10ll * a.W + 3ll * a.R * a.K - 1) /
                              (10ll * a.W + 3ll * a.R * a.K);
        a.n_win = a.w0 == 0 ? kCandRanges
                            : (int)(share < 1 ? 1 : (share > kCandRanges - 1 ? kCandRanges - 1 : share));
    }
    const int n_old = kCandRanges - a.n_win;
    a.span_old = n_old > 0 ? (a.w0 + n_old - 1) / n_old : 0;
    a.span_win = a.n_win > 0 ? (a.len - a.w0 + a.n_win - 1) / a.n_win : 0;
}

Geometry step_geometry(const retopk_config &c, int64_t len, int mode)
{
    Geometry g{};
    // Enough scan blocks to cover the whole chip when every group is scanned;
    // fewer in MODE_SELECT, where the range blocks share the chip.
    const int64_t rows = (int64_t)c.batch * c.n_kv_heads * len;
    const int64_t want = ceil_div(rows, 2 * kScanRowsPerIter);
    // In MODE_SELECT the scan shares the launch with the range blocks and covers
    // only the groups with a fallback head: one scan block per CU, rounded to
    // whole groups of 8 so that the range blocks' XCD placement is kept whichever
    // kind comes first.
    const int cap = mode == MODE_SELECT ? kScanBlocksSelect : kScanBlocksExact;
    g.scan_blocks = (int)(want < cap ? want : cap);
    if (mode == MODE_SELECT) g.scan_blocks = (g.scan_blocks + 7) / 8 * 8;
    // range blocks: whole groups of 8 heads (one head per XCD)
    g.cand_blocks = mode == MODE_SELECT ? (int)((heads_of(c) + 7) / 8 * 8 * kCandRanges) : 0;
    // When the range blocks need more than one block slot per CU, the scan blocks
    // go first, so that they hold a slot on every CU from the start instead of
    // waiting for the range blocks to drain; otherwise the range blocks, which
    // carry the step's critical path, go first.
    g.scan_first = g.cand_blocks > kCUs;
    g.filter_blocks_per_head = (int)ceil_div(len, kFilterRows);
    // Every group scanned, groups of at most 4 heads (the quad row layout) and
    // at least one whole filter region per CU: one k_scan_list block per whole
    // region keeps the region's scores in LDS and writes its local survivors only.
    g.list_mode = (mode == MODE_EXACT || mode == MODE_REFRESH || mode == MODE_COLD) &&
                  c.n_q_heads / c.n_kv_heads <= 4 &&
                  (int64_t)c.batch * c.n_kv_heads * (len / kFilterRows) >= kCUs;
    return g;
}

}  // namespace retopk

namespace {

size_t elem_size(const retopk_config &c) { return c.dtype == RETOPK_BF16 ? 2 : 4; }

template <typename T>
retopk_status alloc(retopk_handle h, T **out, size_t count)
{
    void *p = nullptr;
    size_t bytes = count * sizeof(T);
    if (bytes == 0) bytes = sizeof(T);
    if (hipMalloc(&p, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return RETOPK_ERR_OOM;
    }
    h->allocs.push_back(p);
    if (hipMemset(p, 0, bytes) != hipSuccess) return RETOPK_ERR_HIP;
    *out = (T *)p;
    return RETOPK_OK;
}

StepArgs base_args(const retopk_handle_s *h) { return config_args(h->cfg); }

Geometry make_geometry(const retopk_handle_s *h, int64_t len, int mode)
{
    return step_geometry(h->cfg, len, mode);
}

// Event pair for the next launch of kernel `kid` when profiling is on.
retopk_status timing_for(retopk_handle h, int kid, hipEvent_t *start, hipEvent_t *stop)
{
    *start = *stop = nullptr;
    if (!h->prof) return RETOPK_OK;
    if (h->ev_used / 2 >= (size_t)kProfileMaxLaunches) {
        h->prof_overflow = true;
        return RETOPK_OK;
    }
    while (h->ev.size() < h->ev_used + 2) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return RETOPK_ERR_HIP;
        h->ev.push_back(e);
    }
    *start = h->ev[h->ev_used];
    *stop = h->ev[h->ev_used + 1];
    h->ev_kernel.push_back(kid);
    h->ev_used += 2;
    return RETOPK_OK;
}

retopk_status fail(retopk_handle h)
{
    h->broken = true;
    return RETOPK_ERR_HIP;
}

// Launches one described kernel on s (events attached to its dispatch when
// profiling).
retopk_status launch_desc(retopk_handle h, const KernelDesc &d, int kid, void **args, hipStream_t s)
{
    hipEvent_t start, stop;
    retopk_status st = timing_for(h, kid, &start, &stop);
    if (st != RETOPK_OK) return st;
    hipError_t e = start
        ? hipExtLaunchKernel(d.func, d.grid, d.block, args, d.lds_bytes, s, start, stop, 0)
        : hipLaunchKernel(d.func, d.grid, d.block, args, d.lds_bytes, s);
    return e == hipSuccess ? RETOPK_OK : fail(h);
}

// Launches one step (or one prefill query) in `mode`: SELECT runs k_sim, k_score,
// k_filter, k_final; the other modes k_score (scan only), k_filter, k_final.
// With profiling on, events are attached to each kernel's dispatch.
retopk_status run_step(retopk_handle h, const StepArgs &a, int mode, hipStream_t s)
{
    const Geometry geo = make_geometry(h, a.len, mode);
    const int dt = h->cfg.dtype;
    int kinds[4], n = 0;
    if (mode == MODE_SELECT) kinds[n++] = KERNEL_SIM;
    kinds[n++] = KERNEL_SCORE;
    kinds[n++] = KERNEL_FILTER;
    kinds[n++] = KERNEL_FINAL;
    KernelDesc d[4];
    for (int i = 0; i < n; ++i) describe_kernel(kinds[i], dt, a, geo, &d[i]);
    StepArgs av = a;
    Ws wv = h->w;
    Geometry gv = geo;
    void *args[3] = {&av, &wv, &gv};

    for (int i = 0; i < n; ++i) {
        int kid = KID_FINAL;
        if (kinds[i] == KERNEL_SIM) kid = KID_SIM;
        else if (kinds[i] == KERNEL_SCORE) kid = mode == MODE_SELECT ? KID_SCORE : KID_SCAN;
        else if (kinds[i] == KERNEL_FILTER) kid = KID_FILTER;
        retopk_status st = launch_desc(h, d[i], kid, args, s);
        if (st != RETOPK_OK) return st;
    }
    return RETOPK_OK;
}

// Batched prefill initialisation (bf16): positions u_first .. n-1 of q_tail in
// launches of U positions each, every launch scoring its U x B x Hq virtual
// heads on the matrix cores (k_pf_score) and selecting and inserting them with
// k_filter and k_final, on temporary workspaces.  Returns RETOPK_ERR_OOM, having
// launched nothing, when the workspaces cannot be allocated.
retopk_status prefill_batched(retopk_handle h, const char *q_tail, int32_t n, int32_t u_first,
                              const void *k, const void *v, int64_t prefill_len, hipStream_t s)
{
    const retopk_config &c = h->cfg;
    const int64_t BH = heads_of(c);
    StepArgs a = base_args(h);
    const int64_t NR = a.n_regions, RS = a.row_stride;
    const size_t per_u = (size_t)BH * ((size_t)RS * (8 + 4) + (size_t)NR * 4 + (size_t)kHistBins * 4);
    const int32_t n_eff = n - u_first;
    int64_t U = (int64_t)(kPfWorkspaceBytes / per_u);
    // whole query tiles where the budget allows: U a multiple of kPfCols / gcd(G, kPfCols)
    int gcd = h->G, m = kPfCols;
    while (m) {
        const int r = gcd % m;
        gcd = m;
        m = r;
    }
    const int64_t step = kPfCols / gcd;
    if (U >= step) U -= U % step;
    U = U < 1 ? 1 : (U > n_eff ? n_eff : U);
    void *mem = nullptr;
    if (hipMalloc(&mem, per_u * (size_t)U + 1024) != hipSuccess) {
        (void)hipGetLastError();
        return RETOPK_ERR_OOM;
    }
    Ws w = h->w;
    char *p = (char *)mem;
    w.surv = (uint64_t *)p;
    p += (size_t)U * BH * RS * 8;
    w.scores = (float *)p;
    p += (size_t)U * BH * RS * 4;
    w.hist = (uint32_t *)p;
    p += (size_t)U * BH * kHistBins * 4;
    w.surv_cnt = (uint32_t *)p;
    retopk_status st = RETOPK_OK;
    if (hipMemsetAsync(w.hist, 0, (size_t)U * BH * kHistBins * 4, s) != hipSuccess) st = fail(h);
    const size_t es = elem_size(c);
    for (int32_t u0 = u_first; u0 < n && st == RETOPK_OK; u0 += (int32_t)U) {
        const int32_t Uc = (int32_t)(n - u0 < U ? n - u0 : U);
        StepArgs b = a;
        b.mode = MODE_PREFILL;
        b.U = Uc;
        b.q = q_tail + (size_t)u0 * c.head_dim * es;
        b.q_head_stride = (int64_t)n * c.head_dim;
        b.k = k;
        b.v = v;
        b.len = prefill_len - n + u0 + 1;
        b.out = nullptr;
        b.sel = nullptr;
        b.n_ins = h->n_ins;
        b.insert_slot = (int32_t)(h->n_ins % c.cache_cap);
        b.do_insert = 1;
        const int64_t len_max = b.len + Uc - 1;
        Geometry geo{};
        geo.filter_blocks_per_head = (int)ceil_div(len_max, kFilterRows);
        geo.pf_qtiles = (int)ceil_div((int64_t)h->G * Uc, kPfCols);
        geo.pf_kchunks = (int)ceil_div(len_max, kPfKeys);
        geo.pf_pairs = c.batch * c.n_kv_heads * geo.pf_kchunks;
        void *args[3] = {&b, &w, &geo};
        const int kinds[3] = {KERNEL_PF_SCORE, KERNEL_FILTER, KERNEL_FINAL};
        const int kids[3] = {KID_PF_SCORE, KID_FILTER, KID_FINAL};
        for (int i = 0; i < 3 && st == RETOPK_OK; ++i) {
            KernelDesc d;
            describe_kernel(kinds[i], c.dtype, b, geo, &d);
            st = launch_desc(h, d, kids[i], args, s);
        }
        h->n_ins += Uc;
    }
    // the workspaces are released once the launches that use them are done
    if (hipStreamSynchronize(s) != hipSuccess && st == RETOPK_OK) st = fail(h);
    (void)hipFree(mem);
    return st;
}

// Every call of a handle shares its caches and workspaces, so a call on another
// stream than the previous call's first waits for the work queued there.
retopk_status order_after_last(retopk_handle h, hipStream_t s)
{
    if (!h->has_last || s == h->last_stream) return RETOPK_OK;
    if (!h->order_ev && hipEventCreateWithFlags(&h->order_ev, hipEventDisableTiming) != hipSuccess)
        return fail(h);
    if (hipEventRecord(h->order_ev, h->last_stream) != hipSuccess ||
        hipStreamWaitEvent(s, h->order_ev, 0) != hipSuccess)
        return fail(h);
    return RETOPK_OK;
}

void set_last(retopk_handle h, hipStream_t s)
{
    h->last_stream = s;
    h->has_last = true;
}

retopk_status sync_last(retopk_handle h)
{
    if (hipSetDevice(h->device) != hipSuccess) return RETOPK_ERR_HIP;
    if (hipStreamSynchronize(h->last_stream) != hipSuccess) return fail(h);
    return RETOPK_OK;
}

}  // namespace

extern "C" {

const char *retopk_status_string(retopk_status s)
{
    switch (s) {
    case RETOPK_OK: return "ok";
    case RETOPK_ERR_ARG: return "invalid argument";
    case RETOPK_ERR_UNSUPPORTED: return "unsupported shape";
    case RETOPK_ERR_OOM: return "device out of memory";
    case RETOPK_ERR_HIP: return "HIP runtime error";
    case RETOPK_ERR_STATE: return "call out of order or handle broken";
    case RETOPK_ERR_TOO_LARGE: return "workspace larger than the fixed scratch";
    }
    return "unknown status";
}

const char *retopk_kernel_name(int32_t kernel_id)
{
    return (kernel_id >= 0 && kernel_id < kNumKernels) ? kKernelNames[kernel_id] : nullptr;
}

retopk_status retopk_create(const retopk_config *cfg, retopk_handle *out)
{
    if (!out) return RETOPK_ERR_ARG;
    *out = nullptr;
    retopk_status st = validate_config(cfg);
    if (st != RETOPK_OK) return st;
    retopk_handle h = new (std::nothrow) retopk_handle_s();
    if (!h) return RETOPK_ERR_OOM;
    h->cfg = *cfg;
    h->G = cfg->n_q_heads / cfg->n_kv_heads;
    h->cand_cap = cfg->r * cfg->k + cfg->window;
    h->inv_sqrt_d = (float)(1.0 / std::sqrt((double)cfg->head_dim));
    if (hipGetDevice(&h->device) != hipSuccess) {
        delete h;
        return RETOPK_ERR_HIP;
    }
    const int64_t BH = heads_of(*cfg);
    const int64_t C = cfg->cache_cap, D = cfg->head_dim, K = cfg->k, L = cfg->max_len;
    Ws &w = h->w;
    const int64_t NR = ceil_div(L, kFilterRows), RS = NR * kFilterRows;
    const int64_t NSB = kMaxCache / kSimSlots;
    if ((st = alloc(h, &w.qbar, (size_t)(BH * C * D))) != RETOPK_OK ||
        (st = alloc(h, &w.supp, (size_t)(BH * C * K))) != RETOPK_OK ||
        (st = alloc(h, &w.cnt, (size_t)(BH * C))) != RETOPK_OK ||
        (st = alloc(h, &w.reuse, (size_t)BH)) != RETOPK_OK ||
        (st = alloc(h, &w.topr, (size_t)(BH * NSB * kMaxR))) != RETOPK_OK ||
        (st = alloc(h, &w.topr_rho, (size_t)(BH * NSB * kMaxR))) != RETOPK_OK ||
        (st = alloc(h, &w.topr_cnt, (size_t)(BH * NSB * kMaxR))) != RETOPK_OK ||
        (st = alloc(h, &w.qbar_cur, (size_t)(BH * D))) != RETOPK_OK ||
        (st = alloc(h, &w.path, (size_t)BH)) != RETOPK_OK ||
        (st = alloc(h, &w.scores, (size_t)(BH * RS))) != RETOPK_OK ||
        (st = alloc(h, &w.hist, (size_t)(BH * kHistBins))) != RETOPK_OK ||
        (st = alloc(h, &w.surv, (size_t)(BH * RS))) != RETOPK_OK ||
        (st = alloc(h, &w.surv_cnt, (size_t)(BH * NR))) != RETOPK_OK ||
        (st = alloc(h, &w.cand_ent, (size_t)(BH * kCandRanges * h->cand_cap))) != RETOPK_OK ||
        (st = alloc(h, &w.cand_cnt, (size_t)(BH * kCandRanges))) != RETOPK_OK ||
        (st = alloc(h, &w.stats, (size_t)STAT_COUNT)) != RETOPK_OK ||
        (st = alloc(h, &w.dense_part, (size_t)(BH * ceil_div(cfg->max_len, kDenseRows) *
                                                (cfg->head_dim + 2)))) != RETOPK_OK) {
        retopk_destroy(h);
        return st;
    }
    if (hipDeviceSynchronize() != hipSuccess) {
        retopk_destroy(h);
        return RETOPK_ERR_HIP;
    }
    *out = h;
    return RETOPK_OK;
}

retopk_status retopk_destroy(retopk_handle h)
{
    if (!h) return RETOPK_OK;
    (void)hipSetDevice(h->device);
    if (!h->allocs.empty()) (void)hipDeviceSynchronize();
    for (void *p : h->allocs) (void)hipFree(p);
    for (hipEvent_t e : h->ev) (void)hipEventDestroy(e);
    if (h->order_ev) (void)hipEventDestroy(h->order_ev);
    delete h;
    return RETOPK_OK;
}

retopk_status retopk_decode_step(retopk_handle h, const void *q, const void *k, const void *v,
                                 int64_t len, float *out, int32_t *sel,
                                 const retopk_debug *dbg, void *stream)
{
    if (!h || !q || !k || !v || !out) return RETOPK_ERR_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return RETOPK_ERR_ARG;
    if (len < 1 || len > h->cfg.max_len) return RETOPK_ERR_ARG;
    if (h->broken || len < h->last_len) return RETOPK_ERR_STATE;
    const retopk_config &c = h->cfg;
    const int64_t n_valid = h->n_ins < c.cache_cap ? h->n_ins : c.cache_cap;
    const bool refresh = c.refresh > 0 && h->t_dec > 0 && h->t_dec % c.refresh == 0;
    const int mode = n_valid == 0 ? MODE_COLD : (refresh ? MODE_REFRESH : MODE_SELECT);

    StepArgs a = base_args(h);
    a.mode = mode;
    // Scan-fed candidates pay off when the scan blocks run beside the range blocks
    // from the start (see step_geometry); otherwise the group check would only
    // lengthen the range blocks.
    a.scan_fed = mode == MODE_SELECT && step_geometry(c, len, mode).scan_first ? 1 : 0;
    a.q = q;
    a.k = k;
    a.v = v;
    a.len = len;
    if (mode == MODE_SELECT) range_split(a);
    a.out = out;
    a.sel = sel;
    a.n_ins = h->n_ins;
    a.insert_slot = c.cache_cap > 0 ? (int32_t)(h->n_ins % c.cache_cap) : 0;
    a.do_insert = c.cache_cap > 0 ? 1 : 0;
    if (dbg) {
        a.dbg_path = dbg->path;
        a.dbg_rho = dbg->rho_max;
        a.dbg_ret = dbg->retrieved;
        a.dbg_ncand = dbg->n_cand;
        a.dbg_cand = dbg->cand;
    }
    hipStream_t s = (hipStream_t)stream;
    if (hipSetDevice(h->device) != hipSuccess) return fail(h);
    if (order_after_last(h, s) != RETOPK_OK) return RETOPK_ERR_HIP;
    retopk_status st = run_step(h, a, mode, s);
    if (st != RETOPK_OK) return st;
    set_last(h, s);
    h->last_len = len;
    const int64_t BH = heads_of(c);
    h->steps += 1;
    h->head_steps += (uint64_t)BH;
    if (mode == MODE_REFRESH) h->refresh += (uint64_t)BH;
    if (mode == MODE_COLD) h->cold += (uint64_t)BH;
    if (mode != MODE_SELECT) h->host_scans += (uint64_t)c.batch * c.n_kv_heads;
    if (c.cache_cap > 0) h->n_ins += 1;
    h->t_dec += 1;
    return RETOPK_OK;
}

retopk_status exact_topk_attention(retopk_handle h, const void *q, const void *k,
                                   const void *v, int64_t len, float *out, int32_t *sel,
                                   void *stream)
{
    if (!h || !q || !k || !v || !out) return RETOPK_ERR_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return RETOPK_ERR_ARG;
    if (len < 1 || len > h->cfg.max_len) return RETOPK_ERR_ARG;
    if (h->broken) return RETOPK_ERR_STATE;
    StepArgs a = base_args(h);
    a.mode = MODE_EXACT;
    a.q = q;
    a.k = k;
    a.v = v;
    a.len = len;
    a.out = out;
    a.sel = sel;
    a.do_insert = 0;
    hipStream_t s = (hipStream_t)stream;
    if (hipSetDevice(h->device) != hipSuccess) return fail(h);
    if (order_after_last(h, s) != RETOPK_OK) return RETOPK_ERR_HIP;
    retopk_status st = run_step(h, a, MODE_EXACT, s);
    if (st != RETOPK_OK) return st;
    set_last(h, s);
    return RETOPK_OK;
}

retopk_status retopk_prefill_init(retopk_handle h, const void *q_tail, int32_t n,
                                  const void *k, const void *v, int64_t prefill_len,
                                  void *stream)
{
    if (!h || !k || !v || (n > 0 && !q_tail)) return RETOPK_ERR_ARG;
    if (n < 0 || prefill_len < n || prefill_len > h->cfg.max_len) return RETOPK_ERR_ARG;
    if ((q_tail && !aligned16(q_tail)) || !aligned16(k) || !aligned16(v)) return RETOPK_ERR_ARG;
    if (h->broken) return RETOPK_ERR_STATE;
    const retopk_config &c = h->cfg;
    if (c.cache_cap == 0 || n == 0) return RETOPK_OK;
    hipStream_t s = (hipStream_t)stream;
    if (hipSetDevice(h->device) != hipSuccess) return fail(h);
    if (order_after_last(h, s) != RETOPK_OK) return RETOPK_ERR_HIP;
    // Positions whose slot a later prompt-tail query overwrites (n > C) only
    // advance the insertion count.
    const int32_t u_first = n > c.cache_cap ? n - c.cache_cap : 0;
    h->n_ins += u_first;
    set_last(h, s);
    if (c.dtype == RETOPK_BF16 && n - u_first > 1) {
        const retopk_status st = prefill_batched(h, (const char *)q_tail, n, u_first, k, v,
                                                 prefill_len, s);
        if (st != RETOPK_ERR_OOM) return st;
    }
    const size_t es = elem_size(c);
    for (int32_t u = u_first; u < n; ++u) {
        StepArgs a = base_args(h);
        a.mode = MODE_PREFILL;
        a.q = (const char *)q_tail + (size_t)u * c.head_dim * es;
        a.q_head_stride = (int64_t)n * c.head_dim;
        a.k = k;
        a.v = v;
        a.len = prefill_len - n + u + 1;
        a.out = nullptr;
        a.sel = nullptr;
        a.n_ins = h->n_ins;
        a.insert_slot = (int32_t)(h->n_ins % c.cache_cap);
        a.do_insert = 1;
        retopk_status st = run_step(h, a, MODE_PREFILL, s);
        if (st != RETOPK_OK) return st;
        h->n_ins += 1;
    }
    set_last(h, s);
    return RETOPK_OK;
}

retopk_status retopk_stream_read(const void *src, int64_t bytes, uint32_t *sink, void *stream)
{
    if (!src || !sink || bytes <= 0 || bytes % 16 != 0 || !aligned16(src)) return RETOPK_ERR_ARG;
    launch_stream_read(src, bytes, sink, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? RETOPK_OK : RETOPK_ERR_HIP;
}

retopk_status full_attention(retopk_handle h, const void *q, const void *k, const void *v,
                             int64_t len, float *out, void *stream)
{
    if (!h || !q || !k || !v || !out) return RETOPK_ERR_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return RETOPK_ERR_ARG;
    if (len < 1 || len > h->cfg.max_len) return RETOPK_ERR_ARG;
    if (h->broken) return RETOPK_ERR_STATE;
    StepArgs a = base_args(h);
    a.mode = MODE_EXACT;
    a.q = q;
    a.k = k;
    a.v = v;
    a.len = len;
    a.out = out;
    a.do_insert = 0;
    hipStream_t s = (hipStream_t)stream;
    if (hipSetDevice(h->device) != hipSuccess) return fail(h);
    if (order_after_last(h, s) != RETOPK_OK) return RETOPK_ERR_HIP;
    const Geometry geo = make_geometry(h, len, MODE_EXACT);
    Ws wv = h->w;
    void *args[3] = {&a, &wv, nullptr};
    KernelDesc d;
    describe_kernel(KERNEL_DENSE, h->cfg.dtype, a, geo, &d);
    retopk_status st = launch_desc(h, d, KID_DENSE, args, s);
    if (st != RETOPK_OK) return st;
    describe_kernel(KERNEL_DENSE_MERGE, h->cfg.dtype, a, geo, &d);
    if ((st = launch_desc(h, d, KID_DENSE_MERGE, args, s)) != RETOPK_OK) return st;
    set_last(h, s);
    return RETOPK_OK;
}

retopk_status retopk_stats(retopk_handle h, retopk_stats_t *out)
{
    if (!h || !out) return RETOPK_ERR_ARG;
    retopk_status st = sync_last(h);
    if (st != RETOPK_OK) return st;
    unsigned long long dev[STAT_COUNT];
    if (hipMemcpy(dev, h->w.stats, sizeof(dev), hipMemcpyDeviceToHost) != hipSuccess) return fail(h);
    out->steps = h->steps;
    out->head_steps = h->head_steps;
    out->reuse = dev[STAT_REUSE];
    out->fallback = dev[STAT_FALLBACK];
    out->refresh = h->refresh;
    out->cold = h->cold;
    out->kv_group_scans = dev[STAT_SCANS] + h->host_scans;
    out->cand_sum = dev[STAT_CAND_SUM];
    out->cand_max = dev[STAT_CAND_MAX];
    return RETOPK_OK;
}

retopk_status retopk_get_state(retopk_handle h, float *qbar, int32_t *supp, int32_t *cnt,
                               int64_t *n_inserted, int64_t *t_dec)
{
    if (!h) return RETOPK_ERR_ARG;
    retopk_status st = sync_last(h);
    if (st != RETOPK_OK) return st;
    const retopk_config &c = h->cfg;
    const size_t e = (size_t)heads_of(c) * c.cache_cap;
    if (qbar && e && hipMemcpy(qbar, h->w.qbar, e * c.head_dim * sizeof(float),
                               hipMemcpyDeviceToHost) != hipSuccess)
        return fail(h);
    if (supp && e && hipMemcpy(supp, h->w.supp, e * c.k * sizeof(int32_t),
                               hipMemcpyDeviceToHost) != hipSuccess)
        return fail(h);
    if (cnt && e && hipMemcpy(cnt, h->w.cnt, e * sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess)
        return fail(h);
    if (n_inserted) *n_inserted = h->n_ins;
    if (t_dec) *t_dec = h->t_dec;
    return RETOPK_OK;
}

retopk_status retopk_set_state(retopk_handle h, const float *qbar, const int32_t *supp,
                               const int32_t *cnt, int64_t n_inserted, int64_t t_dec)
{
    if (!h || n_inserted < 0 || t_dec < 0) return RETOPK_ERR_ARG;
    const retopk_config &c = h->cfg;
    const size_t e = (size_t)heads_of(c) * c.cache_cap;
    if (e && (!qbar || !supp || !cnt)) return RETOPK_ERR_ARG;
    for (size_t i = 0; i < e; ++i) {
        if (cnt[i] < 0 || cnt[i] > c.k) return RETOPK_ERR_ARG;
        for (int t = 0; t < cnt[i]; ++t) {
            int32_t x = supp[i * c.k + t];
            if (x < 0 || x >= c.max_len) return RETOPK_ERR_ARG;
        }
        for (int j = 0; j < c.head_dim; ++j)
            if (!std::isfinite(qbar[i * c.head_dim + j])) return RETOPK_ERR_ARG;
    }
    if (h->broken) return RETOPK_ERR_STATE;
    retopk_status st = sync_last(h);
    if (st != RETOPK_OK) return st;
    if (e) {
        if (hipMemcpy(h->w.qbar, qbar, e * c.head_dim * sizeof(float), hipMemcpyHostToDevice) != hipSuccess ||
            hipMemcpy(h->w.supp, supp, e * c.k * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess ||
            hipMemcpy(h->w.cnt, cnt, e * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess)
            return fail(h);
    }
    if (hipMemset(h->w.stats, 0, STAT_COUNT * sizeof(unsigned long long)) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess)
        return fail(h);
    h->n_ins = c.cache_cap > 0 ? n_inserted : 0;
    h->t_dec = t_dec;
    h->last_len = 0;
    h->steps = h->head_steps = h->refresh = h->cold = h->host_scans = 0;
    return RETOPK_OK;
}

retopk_status retopk_profile(retopk_handle h, int32_t enable)
{
    if (!h) return RETOPK_ERR_ARG;
    h->prof = enable != 0;
    if (h->prof) {
        h->ev_used = 0;
        h->ev_kernel.clear();
        h->prof_overflow = false;
    }
    return RETOPK_OK;
}

retopk_status retopk_profile_read(retopk_handle h, int32_t n_kernels, uint64_t *launches,
                                  double *total_ms)
{
    if (!h || n_kernels < 0 || (n_kernels > 0 && (!launches || !total_ms))) return RETOPK_ERR_ARG;
    for (int i = 0; i < n_kernels; ++i) {
        launches[i] = 0;
        total_ms[i] = 0.0;
    }
    retopk_status st = sync_last(h);
    if (st != RETOPK_OK) return st;
    for (size_t i = 0; i < h->ev_used / 2; ++i) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, h->ev[2 * i], h->ev[2 * i + 1]) != hipSuccess) return fail(h);
        const int kid = h->ev_kernel[i];
        if (kid < n_kernels) {
            launches[kid] += 1;
            total_ms[kid] += ms;
        }
    }
    return h->prof_overflow ? RETOPK_ERR_STATE : RETOPK_OK;
}

}  // extern "C"
