// retopk_internal.h -- shared by the host API (retopk_api.hip) and the kernels
// (retopk_kernels.hip).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "retopk.h"

namespace retopk {

// Score histogram used by the full-history selection: bins are the top 11 bits
// of the order-preserving uint32 image of the fp32 score.
constexpr int kHistBins = 2048;
constexpr int kHistShift = 21;

constexpr int kSimThreads = 256;      // k_sim: 64 cached slots per block
constexpr int kSimSlots = 64;
constexpr int kScoreThreads = 512;    // k_score and k_filter blocks
constexpr int kFinalThreads = 512;    // k_final blocks
constexpr int kScanRowsPerIter = 128; // 8 waves x 16 rows
constexpr int kCandRanges = 8;        // index ranges (k_score blocks) per reuse head
constexpr int kCandList = 2048;       // candidates gathered per round in one range block
constexpr int kSegWords = 2048;       // union bitmap segment: 65536 indices
constexpr int kFilterRows = 4096;     // scores filtered per k_filter block
constexpr int kEntCache = 8192;       // final-stage entries staged in LDS
constexpr int kMaxRegions = 4096;     // filter regions per head (max_len <= 16M)
constexpr int kMaxK = 2048;
constexpr int kMaxR = 32;
constexpr int kMaxCache = 4096;
constexpr int kMaxHeads = 2048;       // B * Hq
constexpr int kCUs = 256;               // compute units of the chip
constexpr int kScanBlocksSelect = kCUs; // k_score scan blocks in MODE_SELECT (one per CU)
constexpr int kScanBlocksExact = 2048;  // k_score scan blocks when every head is exact
constexpr int64_t kMaxLen = (int64_t)kMaxRegions * kFilterRows;

// Batched prefill initialisation (bf16): k_pf_score blocks take kPfCols virtual
// queries (one MFMA column each) against kPfKeys keys of one KV group.
constexpr int kPfThreads = 512;
constexpr int kPfCols = 32;
constexpr int kPfKeys = 4096;
constexpr int kPfTiles = 2;           // 16-key tiles per wave per iteration
constexpr int kPfHistStride = kHistBins / 2 + 1;   // padded LDS histogram row (16-bit counts)

// Step modes.  SELECT runs the per-head path rule on the device; the others take
// the exact path for every head.
enum Mode : int {
    MODE_SELECT = 0,    // decode step with a non-empty cache, not a refresh step
    MODE_REFRESH = 1,   // decode step at t_dec in {T_r, 2T_r, ...}
    MODE_COLD = 2,      // decode step with an empty cache
    MODE_EXACT = 3,     // exact_topk_attention: no cache insert, no stats
    MODE_PREFILL = 4    // prefill initialisation: insert only, no output
};

// Path codes (same values as retopk_path).  PATH_REUSE_SCANNED (internal, never
// reported): a reuse head whose KV group is scanned in the same step for another
// head's fallback; its candidates take their scores from that scan.
enum : int8_t { PATH_REUSE = 0, PATH_FALLBACK = 1, PATH_REFRESH = 2, PATH_COLD = 3,
                PATH_REUSE_SCANNED = 4 };

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
    uint8_t *reuse;       // [BH] 1: head bh reuses this step (its rho_max >= tau), set by k_sim,
                          // read by k_score, cleared by k_filter
    int32_t *topr;        // [BH, kMaxCache / kSimSlots, kMaxR] per-k_sim-block Top-R slots
    double *topr_rho;     // [BH, kMaxCache / kSimSlots, kMaxR] their similarities
    int32_t *topr_cnt;    // [BH, kMaxCache / kSimSlots, kMaxR] their support sizes
    float *qbar_cur;      // [BH, d] q_bar of this step
    int8_t *path;         // [BH] path of this step
    float *scores;        // [BH, row_stride] full-history scores of exact heads
    uint32_t *hist;       // [BH, kHistBins] score histogram (zero between steps)
    uint64_t *surv;       // [BH, row_stride] surviving rank entries, region f at f*kFilterRows
    uint32_t *surv_cnt;   // [BH, n_regions] entries in each filter region
    uint64_t *cand_ent;   // [BH, kCandRanges, cand_cap] candidate rank entries per range
    uint32_t *cand_cnt;   // [BH, kCandRanges]
    unsigned long long *stats;  // [STAT_COUNT]
    float *dense_part;    // [BH, n_dense_chunks, d + 2] full attention: o, m, l per chunk
};

// Everything one launch needs (passed by value).
struct StepArgs {
    int B, Hq, Hkv, G, D;
    int64_t max_len;
    int K, M, R, W;
    int cand_cap;
    int n_regions;             // ceil(max_len / kFilterRows): surv_cnt row length
    int n_dense;               // ceil(max_len / kDenseRows): dense_part chunks per head
    int64_t row_stride;        // n_regions * kFilterRows: row length of scores and surv
    float tau;
    int retrieval;             // 0: R most similar entries (Eq. 7); 1: R most recent
    float inv_sqrt_d;          // fl32(1 / sqrt(d))
    int mode;
    int scan_fed;              // MODE_SELECT: the reuse heads of a scanned KV group take
                               // their candidates' scores from the scan (PATH_REUSE_SCANNED)
    const void *q;             // element (b, h, e) at q[(b*Hq + h) * q_head_stride + e]
    int64_t q_head_stride;
    const void *k;
    const void *v;
    int64_t len;               // with U > 1: the length of position 0 of the launch
    // MODE_SELECT: the split of [0, len) into the range blocks' index ranges
    // (range_split): ranges 0 .. kCandRanges-n_win-1 cover [0, w0) in spans of
    // span_old rows, the others the window [w0, len) in spans of span_win
    int64_t w0, span_old, span_win;
    int n_win;
    int U;                     // query positions per launch: 1, or more in the batched
                               // prefill, where virtual head vh = u * B * Hq + bh holds
                               // position u (length len + u, q at + u * d, slot
                               // insert_slot + u) in the workspaces
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
    int scan_blocks;           // scan blocks of k_score (they split the scanned rows)
    int cand_blocks;           // ceil(B * Hq / 8) * 8 * kCandRanges in MODE_SELECT, else 0
    int scan_first;            // k_score's scan blocks come before its range blocks
    int filter_blocks_per_head;
    int list_mode;             // every KV group scanned by k_scan_list, one block per
                               // filter region: k_filter reads local survivors
    // batched prefill (k_pf_score): (KV group, key chunk) pairs, query tiles of
    // kPfCols virtual queries, key chunks of kPfKeys keys per group
    int pf_pairs, pf_qtiles, pf_kchunks;
};

// One kernel of a step, ready to launch (hipLaunchKernel) or to put in a graph
// node: the kernel takes (StepArgs, Ws) when nargs == 2 and (StepArgs, Ws,
// Geometry) when nargs == 3, all by value.
struct KernelDesc {
    const void *func;
    dim3 grid;
    dim3 block;
    unsigned lds_bytes;      // dynamic LDS
    int nargs;
};
enum : int { KERNEL_SIM = 0, KERNEL_SCORE = 1, KERNEL_FILTER = 2, KERNEL_FINAL = 3,
              KERNEL_DENSE = 4, KERNEL_DENSE_MERGE = 5, KERNEL_PF_SCORE = 6 };

// Full (dense) attention: rows per chunk block, and the chunk count for a length.
constexpr int kDenseRows = 1024;
constexpr int kDenseThreads = 512;
constexpr int kMergeThreads = 1024;  // dense merge block: one per query head

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
inline int64_t heads_of(const retopk_config &c) { return (int64_t)c.batch * c.n_q_heads; }

// Host helpers shared by the entry points (retopk_api.hip): the configuration
// check of retopk_create, the launch arguments a configuration fixes (every
// step-dependent field left zero), and the launch geometry of a step.
retopk_status validate_config(const retopk_config *c);
StepArgs config_args(const retopk_config &c);
void range_split(StepArgs &a);
Geometry step_geometry(const retopk_config &c, int64_t len, int mode);

// Fills *k for kernel `which` of a step in a.mode (retopk_kernels.hip).
// dtype: 0 = f32, 1 = bf16.
void describe_kernel(int which, int dtype, const StepArgs &a, const Geometry &geo, KernelDesc *k);
bool shape_supported(int dtype, int d, int g);
// Streaming read of `bytes` at src (a measurement aid; retopk_stream.hip).
void launch_stream_read(const void *src, int64_t bytes, uint32_t *sink, hipStream_t s);

}  // namespace retopk
