// retopk_noalloc.hip -- exact_topk_attention_noalloc: Exact Top-K attention with
// no handle and no device allocation, for callers that cannot allocate (code
// under HIP graph capture, tight serving loops, harnesses that forbid it).
//
// It runs the kernels of exact_topk_attention (full-history scan, survivor
// filter, final selection and Softmax-V) on workspaces carved out of one fixed
// array of device memory, `scratch`, defined below: the library holds one copy
// of it on every GPU it runs on, until the process ends.  All calls on a GPU
// share that GPU's copy, so calls that overlap on one GPU (on different
// streams, or from different host threads) race; each call clears the part that
// must start at zero (the score histograms) with a small fill kernel of its own
// and leaves its other contents behind.
#include "retopk.h"
#include "retopk_internal.h"

#include <mutex>

using namespace retopk;

namespace {

constexpr size_t kScratchBytes = (size_t)RETOPK_NOALLOC_SCRATCH_MB << 20;
constexpr int kMaxDevices = 64;
constexpr size_t kAlign = 256;

// The workspace of every call on a device.  In host code this name stands for
// the array only in hipGetSymbolAddress; kernels get the per-device address.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` on each device

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Workspace layout of one call for B*Hq heads over rows [0, len): full-history
// scores and surviving ranks ([BH, regions * kFilterRows] each), score
// histograms [BH, kHistBins], survivor counts [BH, regions] and candidate
// counts [BH, kCandRanges] (read by the final kernel, unused on the exact path).
// Returns the bytes used; fills *w (when base is not null).
size_t carve(int64_t BH, int64_t len, unsigned char *base, Ws *w)
{
    const int64_t NR = ceil_div(len, kFilterRows), RS = NR * kFilterRows;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        unsigned char *p = base ? base + off : nullptr;
        off += round_up(bytes);
        return p;
    };
    unsigned char *scores = take((size_t)(BH * RS) * sizeof(float));
    unsigned char *surv = take((size_t)(BH * RS) * sizeof(uint64_t));
    unsigned char *hist = take((size_t)(BH * kHistBins) * sizeof(uint32_t));
    unsigned char *surv_cnt = take((size_t)(BH * NR) * sizeof(uint32_t));
    unsigned char *cand_cnt = take((size_t)(BH * kCandRanges) * sizeof(uint32_t));
    if (base && w) {
        *w = Ws{};
        w->scores = (float *)scores;
        w->surv = (uint64_t *)surv;
        w->hist = (uint32_t *)hist;
        w->surv_cnt = (uint32_t *)surv_cnt;
        w->cand_cnt = (uint32_t *)cand_cnt;
    }
    return off;
}

// Zeroes n 32-bit words (a kernel rather than a memset, so that the call can be
// captured in a HIP graph).
__global__ __launch_bounds__(256) void k_clear(uint32_t *p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        p[i] = 0u;
}

// The device address of `scratch` on the current device, looked up once per
// device.
retopk_status scratch_of(void **out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return RETOPK_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return RETOPK_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return RETOPK_ERR_HIP;
        }
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return RETOPK_OK;
}

}  // namespace

extern "C" retopk_status exact_topk_attention_noalloc(const retopk_config *cfg, const void *q,
                                                      const void *k, const void *v, int64_t len,
                                                      float *out, int32_t *sel, void *stream)
{
    retopk_status st = validate_config(cfg);
    if (st != RETOPK_OK) return st;
    if (!q || !k || !v || !out) return RETOPK_ERR_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return RETOPK_ERR_ARG;
    if (len < 1 || len > cfg->max_len) return RETOPK_ERR_ARG;
    const int64_t BH = heads_of(*cfg);
    if (carve(BH, len, nullptr, nullptr) > kScratchBytes) return RETOPK_ERR_TOO_LARGE;

    void *base = nullptr;
    if ((st = scratch_of(&base)) != RETOPK_OK) return st;
    Ws w;
    carve(BH, len, (unsigned char *)base, &w);

    StepArgs a = config_args(*cfg);
    // workspace strides follow this call's length, not max_len
    a.n_regions = (int)ceil_div(len, kFilterRows);
    a.row_stride = (int64_t)a.n_regions * kFilterRows;
    a.mode = MODE_EXACT;
    a.q = q;
    a.k = k;
    a.v = v;
    a.len = len;
    a.out = out;
    a.sel = sel;
    a.do_insert = 0;
    const Geometry geo = step_geometry(*cfg, len, MODE_EXACT);
    hipStream_t s = (hipStream_t)stream;

    // the histograms (and the unused candidate counts) start at zero
    const int64_t nclear = (int64_t)((unsigned char *)w.cand_cnt - (unsigned char *)w.hist) / 4 +
                           BH * kCandRanges;
    const int cblocks = (int)(nclear / 256 + 1 < 1024 ? nclear / 256 + 1 : 1024);
    hipLaunchKernelGGL(k_clear, dim3(cblocks), dim3(256), 0, s, w.hist, nclear);
    if (hipGetLastError() != hipSuccess) return RETOPK_ERR_HIP;

    Geometry gv = geo;
    void *args[3] = {&a, &w, &gv};
    const int kinds[3] = {KERNEL_SCORE, KERNEL_FILTER, KERNEL_FINAL};
    for (int i = 0; i < 3; ++i) {
        KernelDesc d;
        describe_kernel(kinds[i], cfg->dtype, a, geo, &d);
        if (hipLaunchKernel(d.func, d.grid, d.block, args, d.lds_bytes, s) != hipSuccess)
            return RETOPK_ERR_HIP;
    }
    return RETOPK_OK;
}
