// retopk_internal.h -- shared by the host API (retopk_api.hip) and the kernels
// (retopk_kernels.hip).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace retopk {

// Score histogram used by the full-history selection: bins are the top 11 bits
// of the order-preserving uint32 image of the fp32 score.
constexpr int kHistBins = 2048;
constexpr int kHistShift = 21;

constexpr int kScoreThreads = 512;    // k_score and k_filter blocks
constexpr int kSelectThreads = 1024;  // k_select: one block per query head
constexpr int kFinalThreads = 1024;   // k_final: one block per query head
constexpr int kScanRowsPerIter = 128; // 8 waves x 16 rows
constexpr int kCandRows = 512;        // candidates scored per k_score candidate block
constexpr int kFilterRows = 4096;     // scores filtered per k_filter block
constexpr int kBitmapWords = 8192;    // union bitmap segment: 262144 indices
constexpr int kEntCache = 6144;       // final-stage entries staged in LDS
constexpr int kMaxK = 2048;
constexpr int kMaxR = 32;
constexpr int kMaxCache = 4096;

// Step modes.  SELECT runs the per-head path rule on the device; the others take
// the exact path for every head.
enum Mode : int {
    MODE_SELECT = 0,    // decode step with a non-empty cache, not a refresh step
    MODE_REFRESH = 1,   // decode step at t_dec in {T_r, 2T_r, ...}
    MODE_COLD = 2,      // decode step with an empty cache
    MODE_EXACT = 3,     // exact_topk_attention: no cache insert, no stats
    MODE_PREFILL = 4    // prefill initialisation: insert only, no output
};

// Path codes (same values as retopk_path).
enum : int8_t { PATH_REUSE = 0, PATH_FALLBACK = 1, PATH_REFRESH = 2, PATH_COLD = 3 };

// Device counters (uint64) behind retopk_stats.
enum : int {
    STAT_REUSE = 0, STAT_FALLBACK = 1, STAT_SCANS = 2, STAT_CAND_SUM = 3, STAT_CAND_MAX = 4,
    STAT_COUNT = 8
};

// Library-owned device memory.  Head index bh = b * Hq + h.
struct Ws {
    // query-support cache (Eq. 5)
    float *qbar;          // [BH, C, d]
    int32_t *supp;        // [BH, C, K], ascending, -1 padded
    int32_t *cnt;         // [BH, C]
    // per-step workspaces
    float *scores;        // [BH, max_len] full-history scores of exact heads
    uint64_t *surv;       // [BH, max_len] surviving (rank key) entries of exact heads
    uint32_t *hist;       // [BH, kHistBins] score histogram (zero between steps)
    int32_t *cand;        // [BH, cand_cap] candidate set, ascending
    uint64_t *cand_ent;   // [BH, cand_cap] candidate rank keys
    int8_t *path;         // [BH]
    int32_t *n_cand;      // [BH]
    uint32_t *surv_count; // [BH] survivors appended by k_filter (zero between steps)
    unsigned long long *stats;  // [STAT_COUNT]
};

// Everything one launch needs (passed by value).
struct StepArgs {
    int B, Hq, Hkv, G, D;
    int64_t max_len;
    int K, M, R, W;
    int cand_cap;
    float tau;
    float inv_sqrt_d;          // fl32(1 / sqrt(d))
    int mode;
    const void *q;             // element (b, h, e) at q[(b*Hq + h) * q_head_stride + e]
    int64_t q_head_stride;
    const void *k;
    const void *v;
    int64_t len;
    float *out;                // nullable in MODE_PREFILL
    int32_t *sel;              // nullable
    int64_t n_ins;             // insertions before this step
    int32_t insert_slot;       // n_ins mod C (when C > 0)
    int32_t do_insert;
    // diagnostics (nullable)
    int8_t *dbg_path;
    double *dbg_rho;
    int32_t *dbg_ret;
    int32_t *dbg_ncand;
    int32_t *dbg_cand;
};

// Launch geometry chosen on the host.
struct Geometry {
    int scan_chunk_rows;
    int scan_blocks;           // B * Hkv * chunks (0 when the mode never scans)
    int cand_blocks_per_head;  // 0 outside MODE_SELECT
    int filter_blocks_per_head;
};

// Launchers (retopk_kernels.hip).  dtype: 0 = f32, 1 = bf16.
hipError_t launch_select(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                         hipStream_t s);
hipError_t launch_score(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                        hipStream_t s);
hipError_t launch_filter(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                         hipStream_t s);
hipError_t launch_final(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                        hipStream_t s);
bool shape_supported(int dtype, int d, int g);

}  // namespace retopk
