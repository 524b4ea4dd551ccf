// retopk_kernels.hip -- gfx950 (CDNA4) kernels of the ReTopK decode step.
//
// One decode step is four launches on the caller's stream, and blocks never wait
// on each other inside a launch (every hand-over is a kernel boundary):
//   k_sim     cosine similarity of q_bar to every cached query (Eq. 5, Eq. 6),
//             64 cache slots per block, plus per-block maxima of rho.
//   k_score   (a) full-history QK scan of every KV group with an exact head
//             (Eq. 4): one key-row load serves the G query heads of the group, and
//             each block adds its scores to a per-head histogram;
//             (b) for every query head, kCandRanges blocks each own one index range:
//             they apply the path rule (Eq. 13), take the Top-R cache entries
//             (Eq. 7), form the range's part of the candidate set (Eq. 8-9) through
//             an LDS bitmap and score those keys (Eq. 10).
//   k_filter  per exact head, the scores at or above the histogram bin that holds
//             the K-th largest, compacted in index order.
//   k_final   kFinalSlices blocks per head: each selects the Top-K of the head's
//             candidates (Eq. 11) or surviving scores (Eq. 1) by radix select on
//             64-bit ranks, then aggregates one slice of the head dimension of
//             Softmax-V (Eq. 12); slice 0 writes the support and inserts into the
//             cache (Sec. 3.4).
// Exact Top-K attention alone is k_score (scan only) + k_filter + k_final.
//
// Ranking is on the fp32 scaled score fl32(q.k) * fl32(1/sqrt d) with ties to the
// lower index: every entry carries a 64-bit rank (score key << 32 | ~index), and
// ranks are distinct.
#include "retopk_internal.h"

#include <hip/hip_ext.h>

namespace retopk {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Scalar helpers
// ---------------------------------------------------------------------------

// Order-preserving image of an fp32 score (finite inputs); -0.0 maps like +0.0.
__device__ __forceinline__ uint32_t ord_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_score(uint32_t k)
{
    uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// Larger rank = higher score, or equal score and lower index.
__device__ __forceinline__ uint64_t rank_of(float s, uint32_t idx)
{
    return ((uint64_t)ord_key(s) << 32) | (uint64_t)(0xFFFFFFFFu - idx);
}
__device__ __forceinline__ uint32_t rank_index(uint64_t r) { return 0xFFFFFFFFu - (uint32_t)r; }
__device__ __forceinline__ uint32_t rank_key(uint64_t r) { return (uint32_t)(r >> 32); }

__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xFFFF0000u); }

template <typename T> __device__ __forceinline__ double elem_f64(const T *p, int i);
template <> __device__ __forceinline__ double elem_f64<float>(const float *p, int i)
{
    return (double)p[i];
}
template <> __device__ __forceinline__ double elem_f64<uint16_t>(const uint16_t *p, int i)
{
    return (double)__uint_as_float((uint32_t)p[i] << 16);
}

// ---------------------------------------------------------------------------
// Cross-lane helpers (DPP inside a quad of lanes; shuffles elsewhere)
// ---------------------------------------------------------------------------

constexpr int kQuadXor1 = 0xB1;   // quad_perm:[1,0,3,2]
constexpr int kQuadXor2 = 0x4E;   // quad_perm:[2,3,0,1]

template <int CTRL> __device__ __forceinline__ float dpp_f32(float x)
{
    return __builtin_bit_cast(float,
        __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

template <int CTRL> __device__ __forceinline__ double dpp_f64(double x)
{
    uint64_t u = __builtin_bit_cast(uint64_t, x);
    int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, true);
    int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, true);
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

// Sum over the 4 lanes of a quad; every lane of the quad gets the same value.
__device__ __forceinline__ float quad_sum(float x)
{
    x += dpp_f32<kQuadXor1>(x);
    x += dpp_f32<kQuadXor2>(x);
    return x;
}
__device__ __forceinline__ double quad_sum(double x)
{
    x += dpp_f64<kQuadXor1>(x);
    x += dpp_f64<kQuadXor2>(x);
    return x;
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v)
{
    const int l = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        uint32_t t = __shfl_up(v, o);
        if (l >= o) v += t;
    }
    return v;
}

// Block reductions.  All threads must call them; every thread gets the same
// result (fixed combination order).  red: NT/64 scratch slots.
template <int NT, typename V, typename Op>
__device__ __forceinline__ V block_reduce(V v, V *red, Op op)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = op(v, __shfl_xor(v, o));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    V t = red[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) t = op(t, red[w]);
    __syncthreads();
    return t;
}

// Exclusive prefix sum over the block; *total receives the block sum.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *red, uint32_t *total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t incl = wave_incl_scan(v);
    if (lane == 63) red[wave] = incl;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
        uint32_t x = red[w];
        if (w < wave) before += x;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return before + incl - v;
}

// ---------------------------------------------------------------------------
// Row geometry.  A row of D elements of type T is split over the 4 lanes of a
// quad: lane p holds the 16-byte vectors s*4 + p, s = 0 .. NV-1.  One wave covers
// 16 rows per pass, and each load instruction reads 64 contiguous bytes per row.
// ---------------------------------------------------------------------------

template <typename T, int D> struct RowT {
    static constexpr int kBytes = D * (int)sizeof(T);
    static constexpr int kNV = kBytes / 64;
    static constexpr int kEPV = 16 / (int)sizeof(T);
};

template <typename T> struct Dot;
template <> struct Dot<uint16_t> {
    // 8 bf16 products accumulated in fp32 with v_dot2_f32_bf16.
    static __device__ __forceinline__ float f(uint4 k, uint4 q, float acc)
    {
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, k.x),
                                              __builtin_bit_cast(bf16x2_t, q.x), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, k.y),
                                              __builtin_bit_cast(bf16x2_t, q.y), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, k.z),
                                              __builtin_bit_cast(bf16x2_t, q.z), acc, false);
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, k.w),
                                              __builtin_bit_cast(bf16x2_t, q.w), acc, false);
        return acc;
    }
    static __device__ __forceinline__ void axpy(uint4 v, float w, float *acc)
    {
        acc[0] += w * bf16_lo(v.x); acc[1] += w * bf16_hi(v.x);
        acc[2] += w * bf16_lo(v.y); acc[3] += w * bf16_hi(v.y);
        acc[4] += w * bf16_lo(v.z); acc[5] += w * bf16_hi(v.z);
        acc[6] += w * bf16_lo(v.w); acc[7] += w * bf16_hi(v.w);
    }
};
template <> struct Dot<float> {
    static __device__ __forceinline__ float f(uint4 k, uint4 q, float acc)
    {
        acc = fmaf(__uint_as_float(k.x), __uint_as_float(q.x), acc);
        acc = fmaf(__uint_as_float(k.y), __uint_as_float(q.y), acc);
        acc = fmaf(__uint_as_float(k.z), __uint_as_float(q.z), acc);
        acc = fmaf(__uint_as_float(k.w), __uint_as_float(q.w), acc);
        return acc;
    }
    static __device__ __forceinline__ void axpy(uint4 v, float w, float *acc)
    {
        acc[0] += w * __uint_as_float(v.x); acc[1] += w * __uint_as_float(v.y);
        acc[2] += w * __uint_as_float(v.z); acc[3] += w * __uint_as_float(v.w);
    }
};

// Reduce-scatter inside a quad: lane p of the quad holds partial sums a0..a3 of
// four dot products; on return it holds the full (4-lane) sum of dot product p.
// Two butterfly steps: at each one a lane keeps the half of its values whose
// index bit matches its own lane bit and sends the other half to its partner.
__device__ __forceinline__ float quad_transpose_sum(float a0, float a1, float a2, float a3, int p)
{
    const bool b0 = (p & 1) != 0, b1 = (p & 2) != 0;
    const float keep0 = b0 ? a1 : a0, send0 = b0 ? a0 : a1;
    const float keep1 = b0 ? a3 : a2, send1 = b0 ? a2 : a3;
    const float r0 = keep0 + dpp_f32<kQuadXor1>(send0);   // dot 0 + b0
    const float r1 = keep1 + dpp_f32<kQuadXor1>(send1);   // dot 2 + b0
    const float keep = b1 ? r1 : r0, send = b1 ? r0 : r1;
    return keep + dpp_f32<kQuadXor2>(send);                // dot 2*b1 + b0
}

// Full scores of a G-head group after each lane of a quad accumulated its quarter
// of every row: lane p returns the scores of heads p and p + 4 (when they exist).
template <int G>
__device__ __forceinline__ void group_scores(const float (&acc)[G], int p, float &s_lo, float &s_hi)
{
    if constexpr (G == 1) {
        s_lo = quad_sum(acc[0]);
        s_hi = 0.0f;
    } else if constexpr (G == 2) {
        const bool b0 = (p & 1) != 0;
        const float r = (b0 ? acc[1] : acc[0]) + dpp_f32<kQuadXor1>(b0 ? acc[0] : acc[1]);
        s_lo = r + dpp_f32<kQuadXor2>(r);
        s_hi = 0.0f;
    } else if constexpr (G == 4) {
        s_lo = quad_transpose_sum(acc[0], acc[1], acc[2], acc[3], p);
        s_hi = 0.0f;
    } else {
        s_lo = quad_transpose_sum(acc[0], acc[1], acc[2], acc[3], p);
        s_hi = quad_transpose_sum(acc[4], acc[5], acc[6], acc[7], p);
    }
}

// ---------------------------------------------------------------------------
// q_bar = fl32(q / ||q||_2), norm in float64 (Eq. 5, Eq. 6)
// ---------------------------------------------------------------------------

template <typename T, int D, int NT>
__device__ void block_qbar(const T *q, float *s_qbar, double *red)
{
    static_assert(NT >= D, "one thread per element");
    const int t = threadIdx.x;
    double x = t < D ? elem_f64<T>(q, t) : 0.0;
    double ss = block_reduce<NT>(x * x, red, [](double a, double b) { return a + b; });
    double nrm = sqrt(ss);
    if (t < D) s_qbar[t] = nrm > 0.0 ? (float)(x / nrm) : 0.0f;
    __syncthreads();
}


// ---------------------------------------------------------------------------
// k_sim: rho for 64 cache slots per block (Eq. 6)
// ---------------------------------------------------------------------------

template <typename T, int D>
__global__ __launch_bounds__(kSimThreads) void k_sim(StepArgs a, Ws w)
{
    constexpr int NT = kSimThreads;
    __shared__ float s_qbar[D];
    __shared__ double s_red[NT / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3;
    const int M = a.M;
    const int nsb = (M + kSimSlots - 1) / kSimSlots;
    const int bh = blockIdx.x / nsb, sb = blockIdx.x % nsb;
    const int n_valid = (int)(a.n_ins < (int64_t)M ? a.n_ins : (int64_t)M);

    block_qbar<T, D, NT>((const T *)a.q + (int64_t)bh * a.q_head_stride, s_qbar, s_red);
    if (sb == 0)
        for (int t = tid; t < D; t += NT) w.qbar_cur[(int64_t)bh * D + t] = s_qbar[t];

    // 16 slots per wave, 4 lanes per cached row of D floats.
    const int slot = sb * kSimSlots + wave * 16 + (lane >> 2);
    const float4 *crow = (const float4 *)(w.qbar + ((int64_t)bh * M + (slot < n_valid ? slot : 0)) * D);
    float4 c[D / 16];
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
        c[s] = slot < n_valid ? crow[s * 4 + p] : make_float4(0.f, 0.f, 0.f, 0.f);
    double acc = 0.0;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
        const float *qq = &s_qbar[(s * 4 + p) * 4];
        acc += (double)c[s].x * (double)qq[0];
        acc += (double)c[s].y * (double)qq[1];
        acc += (double)c[s].z * (double)qq[2];
        acc += (double)c[s].w * (double)qq[3];
    }
    acc = quad_sum(acc);
    if (slot < n_valid && p == 0) w.rho[(int64_t)bh * M + slot] = acc;
    const double bmax = block_reduce<NT>(slot < n_valid ? acc : -INFINITY, s_red,
                                         [](double x, double y) { return fmax(x, y); });
    if (tid == 0) w.rho_bmax[(int64_t)bh * (kMaxCache / kSimSlots) + sb] = bmax;
}

// ---------------------------------------------------------------------------
// k_score
// ---------------------------------------------------------------------------

// LDS of k_score: the scan blocks' histograms, or a range block's rho array,
// which later holds the union bitmap segment and the candidate list.
template <int G>
struct ScoreLds {
    static constexpr int kScan = G * kHistBins * 4;
    static constexpr int kRho = 8 * kMaxCache;
    static constexpr int kSeg = kSegWords * 4 + kCandList * 4;
    static constexpr int kCand = kRho > kSeg ? kRho : kSeg;
    static constexpr int kBytes = kScan > kCand ? kScan : kCand;
};

// Scan block: scores of rows [chunk*rows, ...) of KV head (b, g) for the group's
// exact heads, written to `scores` and counted in the per-head histogram.
template <typename T, int D, int G>
__device__ void scan_block(const StepArgs &a, const Ws &w, const Geometry &geo, unsigned char *lds)
{
    using R = RowT<T, D>;
    __shared__ uint32_t s_exmask;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int chunks = geo.scan_blocks / (a.B * a.Hkv);
    const int bg = blockIdx.x / chunks, chunk = blockIdx.x % chunks;
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    const int bh0 = b * a.Hq + g * G;

    if (tid == 0) {
        uint32_t m = (1u << G) - 1u;
        if (a.mode == MODE_SELECT) {
            // Eq. 13: a head is exact iff rho_max < tau (rho_max from k_sim's block maxima).
            const int nsb = (a.M + kSimSlots - 1) / kSimSlots;
            m = 0u;
            for (int j = 0; j < G; ++j) {
                double mx = -INFINITY;
                for (int sb = 0; sb < nsb; ++sb)
                    mx = fmax(mx, w.rho_bmax[(int64_t)(bh0 + j) * (kMaxCache / kSimSlots) + sb]);
                if (mx < (double)a.tau) m |= 1u << j;
            }
        }
        s_exmask = m;
    }
    __syncthreads();
    const uint32_t exmask = s_exmask;
    if (exmask == 0) return;
    const int64_t row0 = (int64_t)chunk * geo.scan_chunk_rows;
    if (row0 >= a.len) return;
    if (a.mode == MODE_SELECT && chunk == 0 && tid == 0) atomicAdd(&w.stats[STAT_SCANS], 1ull);

    uint32_t *s_hist = (uint32_t *)lds;
    for (int i = tid; i < G * kHistBins; i += kScoreThreads) s_hist[i] = 0u;
    __syncthreads();

    uint4 qv[G][R::kNV];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)(bh0 + j) * a.q_head_stride);
#pragma unroll
        for (int s = 0; s < R::kNV; ++s) qv[j][s] = qr[s * 4 + p];
    }
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    const int64_t row_end = (row0 + geo.scan_chunk_rows < a.len) ? row0 + geo.scan_chunk_rows : a.len;

    for (int64_t base = row0; base < row_end; base += 2 * kScanRowsPerIter) {
        uint4 kv[2][R::kNV];
        int64_t row[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            row[u] = base + u * kScanRowsPerIter + wave * 16 + rl;
            if (row[u] < row_end) {
                const uint4 *rp = (const uint4 *)(kbase + row[u] * D);
#pragma unroll
                for (int s = 0; s < R::kNV; ++s) kv[u][s] = rp[s * 4 + p];
            } else {
#pragma unroll
                for (int s = 0; s < R::kNV; ++s) kv[u][s] = make_uint4(0u, 0u, 0u, 0u);
            }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            float acc[G];
#pragma unroll
            for (int j = 0; j < G; ++j) {
                float s0 = 0.0f;
#pragma unroll
                for (int s = 0; s < R::kNV; ++s) s0 = Dot<T>::f(kv[u][s], qv[j][s], s0);
                acc[j] = s0;
            }
            float sc_lo, sc_hi;
            group_scores<G>(acc, p, sc_lo, sc_hi);
            if (row[u] < row_end) {
#pragma unroll
                for (int jj = 0; jj < (G + 3) / 4; ++jj) {
                    const int j = jj * 4 + (G == 1 ? 0 : (G == 2 ? (p & 1) : p));
                    const bool mine = G == 1 ? p == 0 : (G == 2 ? p < 2 : true);
                    if (mine && ((exmask >> j) & 1u)) {
                        const float sc = (jj == 0 ? sc_lo : sc_hi) * a.inv_sqrt_d;
                        w.scores[(int64_t)(bh0 + j) * a.row_stride + row[u]] = sc;
                        atomicAdd(&s_hist[j * kHistBins + (ord_key(sc) >> kHistShift)], 1u);
                    }
                }
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < G * kHistBins; i += kScoreThreads) {
        const int j = i / kHistBins;
        if ((exmask >> j) & 1u) {
            uint32_t c = s_hist[i];
            if (c) atomicAdd(&w.hist[(int64_t)(bh0 + j) * kHistBins + (i % kHistBins)], c);
        }
    }
}

// Range block s of head bh: path rule, Top-R, the head's candidates inside index
// range s, and their scores.  Entries go to region (bh, s) in index order.
template <typename T, int D>
__device__ void range_block(const StepArgs &a, const Ws &w, int cb, unsigned char *lds)
{
    using R = RowT<T, D>;
    constexpr int NT = kScoreThreads;
    __shared__ double s_red64[NT / 64];
    __shared__ uint32_t s_red32[NT / 64];
    __shared__ int32_t s_ret[kMaxR];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int bh = cb / kCandRanges, s = cb % kCandRanges;
    const int M = a.M;
    const int n_valid = (int)(a.n_ins < (int64_t)M ? a.n_ins : (int64_t)M);
    double *s_rho = (double *)lds;

    // rho of every valid slot (written by k_sim), rho_max and the path (Eq. 13).
    double mx = -INFINITY;
    for (int i = tid; i < n_valid; i += NT) {
        const double r = w.rho[(int64_t)bh * M + i];
        s_rho[i] = r;
        mx = fmax(mx, r);
    }
    mx = block_reduce<NT>(mx, s_red64, [](double x, double y) { return fmax(x, y); });
    const int8_t path = mx < (double)a.tau ? PATH_FALLBACK : PATH_REUSE;
    const int nret = path == PATH_REUSE ? (a.R < n_valid ? a.R : n_valid) : 0;
    if (s == 0 && tid == 0) {
        w.path[bh] = path;
        if (a.dbg_path) a.dbg_path[bh] = path;
        if (a.dbg_rho) a.dbg_rho[bh] = mx;
        atomicAdd(&w.stats[path == PATH_REUSE ? STAT_REUSE : STAT_FALLBACK], 1ull);
    }
    if (path != PATH_REUSE) {
        if (s == 0 && a.dbg_ret)
            for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = -1;
        return;
    }

    // Eq. 7: slot i is the rank-th retrieved entry, rank = number of slots that are
    // more similar, or equally similar and newer (age (n_ins-1-slot) mod C).
    const int age0 = (int)(((a.n_ins - 1) % M + M) % M);
    for (int i = tid; i < n_valid; i += NT) {
        const double ri = s_rho[i];
        const int ai = (age0 - i + M) % M;
        int rank = 0;
        for (int j = 0; j < n_valid && rank < nret; ++j) {
            const double rj = s_rho[j];
            const int aj = (age0 - j + M) % M;
            rank += (rj > ri || (rj == ri && aj < ai)) ? 1 : 0;
        }
        if (rank < nret) s_ret[rank] = i;
    }
    __syncthreads();
    if (s == 0 && a.dbg_ret)
        for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = i < nret ? s_ret[i] : -1;

    // Eq. 8-9 restricted to this block's index range [lo, hi).
    const int64_t len = a.len;
    const int64_t span = (len + kCandRanges - 1) / kCandRanges;
    const int64_t lo = (int64_t)s * span;
    const int64_t hi = lo + span < len ? lo + span : len;
    const int64_t w0 = len - a.W > 0 ? len - a.W : 0;
    uint32_t *bitmap = (uint32_t *)lds;                    // reuses the rho space
    int32_t *list = (int32_t *)(lds + kSegWords * 4);
    uint64_t *ents = w.cand_ent + ((int64_t)bh * kCandRanges + s) * a.cand_cap;
    const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    uint4 qv[R::kNV];
    {
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)bh * a.q_head_stride);
#pragma unroll
        for (int v = 0; v < R::kNV; ++v) qv[v] = qr[v * 4 + p];
    }
    __syncthreads();   // s_rho is dead from here on

    int total = 0;
    for (int64_t seg = lo; seg < hi; seg += (int64_t)kSegWords * 32) {
        const int64_t seg_hi = seg + (int64_t)kSegWords * 32 < hi ? seg + (int64_t)kSegWords * 32 : hi;
        const int nwords = (int)((seg_hi - seg + 31) >> 5);
        for (int i = tid; i < nwords; i += NT) bitmap[i] = 0u;
        __syncthreads();
        for (int r = 0; r < nret; ++r) {
            const int64_t e = (int64_t)bh * M + s_ret[r];
            const int32_t *sp = w.supp + e * a.K;
            const int c = w.cnt[e];
            for (int t = tid; t < c; t += NT) {
                const int64_t x = sp[t];
                if (x >= seg && x < seg_hi) atomicOr(&bitmap[(x - seg) >> 5], 1u << ((x - seg) & 31));
            }
        }
        for (int64_t x = (w0 > seg ? w0 : seg) + tid; x < seg_hi; x += NT)
            atomicOr(&bitmap[(x - seg) >> 5], 1u << ((x - seg) & 31));
        __syncthreads();
        const int wpt = (nwords + NT - 1) / NT;
        const int wb = tid * wpt < nwords ? tid * wpt : nwords;
        const int we = wb + wpt < nwords ? wb + wpt : nwords;
        uint32_t mine = 0;
        for (int i = wb; i < we; ++i) mine += __popc(bitmap[i]);
        uint32_t seg_total;
        const uint32_t first = block_excl_scan<NT>(mine, s_red32, &seg_total);
        for (uint32_t rb = 0; rb < seg_total; rb += kCandList) {
            // emit this round's candidates (ascending) into the LDS list
            uint32_t pos = first;
            for (int i = wb; i < we && pos < rb + kCandList; ++i) {
                uint32_t bits = bitmap[i];
                while (bits) {
                    const int bit = __ffs(bits) - 1;
                    bits &= bits - 1u;
                    if (pos >= rb && pos < rb + kCandList)
                        list[pos - rb] = (int32_t)(seg + (int64_t)i * 32 + bit);
                    ++pos;
                }
            }
            __syncthreads();
            const int nr = (int)(seg_total - rb < (uint32_t)kCandList ? seg_total - rb : kCandList);
            // Eq. 10 on this round: 4 lanes per key row, two rows per lane in flight.
            for (int base = 0; base < nr; base += 2 * kScanRowsPerIter) {
                uint4 kv[2][R::kNV];
                int ci[2], cidx[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    ci[u] = base + u * kScanRowsPerIter + wave * 16 + rl;
                    cidx[u] = ci[u] < nr ? list[ci[u]] : 0;
                    const uint4 *rp = (const uint4 *)(kbase + (int64_t)cidx[u] * D);
#pragma unroll
                    for (int v = 0; v < R::kNV; ++v)
                        kv[u][v] = ci[u] < nr ? rp[v * 4 + p] : make_uint4(0u, 0u, 0u, 0u);
                }
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    float s0 = 0.0f;
#pragma unroll
                    for (int v = 0; v < R::kNV; ++v) s0 = Dot<T>::f(kv[u][v], qv[v], s0);
                    s0 = quad_sum(s0);
                    if (p == 0 && ci[u] < nr)
                        ents[total + rb + ci[u]] = rank_of(s0 * a.inv_sqrt_d, (uint32_t)cidx[u]);
                }
            }
            __syncthreads();
        }
        total += (int)seg_total;
    }
    if (tid == 0) w.cand_cnt[(int64_t)bh * kCandRanges + s] = (uint32_t)total;
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kScoreThreads) void k_score(StepArgs a, Ws w, Geometry geo)
{
    __shared__ __attribute__((aligned(16))) unsigned char lds[ScoreLds<G>::kBytes];
    if ((int)blockIdx.x < geo.scan_blocks)
        scan_block<T, D, G>(a, w, geo, lds);
    else
        range_block<T, D>(a, w, (int)blockIdx.x - geo.scan_blocks, lds);
}

// ---------------------------------------------------------------------------
// k_filter: survivors of every exact head, compacted in index order per block
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kScoreThreads) void k_filter(StepArgs a, Ws w, Geometry geo)
{
    constexpr int NT = kScoreThreads;
    constexpr int EPT = kFilterRows / NT;   // 8 consecutive scores per thread
    static_assert(NT * 4 == kHistBins, "4 histogram bins per thread");
    static_assert(EPT == 8, "two float4 per thread");
    __shared__ uint32_t s_red[NT / 64];
    __shared__ uint32_t s_bstar;
    const int tid = threadIdx.x;
    const int bh = blockIdx.x / geo.filter_blocks_per_head;
    const int f = blockIdx.x % geo.filter_blocks_per_head;
    if (a.mode == MODE_SELECT && w.path[bh] == PATH_REUSE) return;

    // The bin b* that holds the kn-th largest score: the largest b with
    // count(bins >= b) >= kn.  Thread t holds bins 2047-4t .. 2044-4t.
    {
        const uint32_t kn = (uint32_t)(a.K < a.len ? a.K : a.len);
        const uint32_t *hist = w.hist + (int64_t)bh * kHistBins;
        uint32_t c[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) c[j] = hist[kHistBins - 1 - 4 * tid - j];
        uint32_t all;
        uint32_t above = block_excl_scan<NT>(c[0] + c[1] + c[2] + c[3], s_red, &all);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (above < kn && above + c[j] >= kn) s_bstar = (uint32_t)(kHistBins - 1 - 4 * tid - j);
            above += c[j];
        }
        __syncthreads();
    }
    const uint32_t kmin = s_bstar << kHistShift;
    const int64_t i0 = (int64_t)f * kFilterRows + (int64_t)tid * EPT;
    const float4 *src = (const float4 *)(w.scores + (int64_t)bh * a.row_stride + i0);
    const float4 v0 = src[0], v1 = src[1];
    const float sv[EPT] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint32_t keep = 0, n = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const bool k = i0 + e < a.len && ord_key(sv[e]) >= kmin;
        keep |= (uint32_t)k << e;
        n += k ? 1u : 0u;
    }
    uint32_t total;
    uint32_t pos = block_excl_scan<NT>(n, s_red, &total);
    uint64_t *dst = w.surv + (int64_t)bh * a.row_stride + (int64_t)f * kFilterRows;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
        if ((keep >> e) & 1u) dst[pos++] = rank_of(sv[e], (uint32_t)(i0 + e));
    if (tid == 0) w.surv_cnt[(int64_t)bh * a.n_regions + f] = total;
}

// ---------------------------------------------------------------------------
// k_final
// ---------------------------------------------------------------------------

template <int D, int NT>
struct FinalSmem {
    uint64_t ent[kEntCache];        // the head's entries in index order, when they fit
    uint64_t sel[kMaxK];            // selected (index << 32 | score key), index order
    float wgt[kMaxK];
    uint32_t pref[kMaxRegions + 1]; // region prefix counts
    uint32_t hist[kHistBins];
    float part[NT / 64][D / kFinalSlices];
    float qbar[D];
    double red64[NT / 64];
    float red32[NT / 64];
    uint32_t redu[NT / 64];
    uint32_t found_digit, found_above, found_cnt;
};

// Entries of one head, spread over regions of a fixed stride, read in order.
struct Regions {
    const uint64_t *base;
    int64_t stride;
    int n;
    const uint64_t *staged;   // LDS copy or nullptr
    const uint32_t *pref;
    int nreg;
    __device__ uint64_t get(int j) const
    {
        if (staged) return staged[j];
        int lo = 0, hi = nreg - 1;   // last region r with pref[r] <= j
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int)pref[mid] <= j) lo = mid; else hi = mid - 1;
        }
        return base[(int64_t)lo * stride + (j - (int)pref[lo])];
    }
};

// Radix select over distinct 64-bit ranks with 11-bit digits, most significant
// first.  On return the top min(K, n) entries are exactly those with
// (rank & mask) >= prefix (mask == 0 selects everything).
template <int D, int NT>
__device__ void radix_threshold(const Regions &rg, int K, FinalSmem<D, NT> &sm, uint64_t &prefix,
                                uint64_t &mask)
{
    const int tid = threadIdx.x;
    prefix = 0;
    mask = 0;
    if (rg.n <= K) return;
    uint32_t k_rem = (uint32_t)K;
    for (int shift = 53; ; shift -= 11) {
        const int sh = shift > 0 ? shift : 0;
        const int width = shift > 0 ? 11 : 11 + shift;
        const uint32_t nb = 1u << width;
        for (uint32_t i = tid; i < nb; i += NT) sm.hist[i] = 0u;
        __syncthreads();
        for (int j = tid; j < rg.n; j += NT) {
            const uint64_t e = rg.get(j);
            if ((e & mask) == prefix) atomicAdd(&sm.hist[(uint32_t)(e >> sh) & (nb - 1u)], 1u);
        }
        __syncthreads();
        // thread t covers digits nb-1-4t .. nb-4-4t (descending)
        uint32_t c[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int dgt = (int)nb - 1 - 4 * tid - j;
            c[j] = dgt >= 0 ? sm.hist[dgt] : 0u;
        }
        uint32_t all;
        uint32_t above = block_excl_scan<NT>(c[0] + c[1] + c[2] + c[3], sm.redu, &all);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (above < k_rem && above + c[j] >= k_rem) {
                sm.found_digit = nb - 1u - 4u * tid - j;
                sm.found_above = above;
                sm.found_cnt = c[j];
            }
            above += c[j];
        }
        __syncthreads();
        k_rem -= sm.found_above;
        prefix |= (uint64_t)sm.found_digit << sh;
        mask |= (uint64_t)(nb - 1u) << sh;
        const bool done = sm.found_cnt == k_rem || sh == 0;
        __syncthreads();
        if (done) break;
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kFinalThreads) void k_final(StepArgs a, Ws w)
{
    constexpr int NT = kFinalThreads;
    constexpr int NW = NT / 64;
    constexpr int DS = D / kFinalSlices;                 // elements per slice
    constexpr int SB = DS * (int)sizeof(T);              // bytes per slice row
    constexpr int LPR = SB / 16;                         // lanes per slice row
    constexpr int RPW = 64 / LPR;                        // rows per wave instruction
    constexpr int EPV = 16 / (int)sizeof(T);
    static_assert(SB % 16 == 0 && LPR >= 1 && LPR <= 64, "slice geometry");
    __shared__ FinalSmem<D, NT> sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.x / kFinalSlices, slice = blockIdx.x % kFinalSlices;
    const bool writes_out = a.out != nullptr && a.mode != MODE_PREFILL;
    if (slice != 0 && !writes_out) return;

    if (slice == 0 && (a.mode == MODE_REFRESH || a.mode == MODE_COLD)) {
        const int8_t code = a.mode == MODE_REFRESH ? PATH_REFRESH : PATH_COLD;
        if (tid == 0) {
            if (a.dbg_path) a.dbg_path[bh] = code;
            if (a.dbg_rho) a.dbg_rho[bh] = __builtin_nan("");
        }
        if (a.dbg_ret)
            for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = -1;
    }
    const bool reuse = a.mode == MODE_SELECT && w.path[bh] == PATH_REUSE;

    // Region layout of this head's entries.
    Regions rg;
    const uint32_t *cnts;
    if (reuse) {
        rg.base = w.cand_ent + (int64_t)bh * kCandRanges * a.cand_cap;
        rg.stride = a.cand_cap;
        rg.nreg = kCandRanges;
        cnts = w.cand_cnt + (int64_t)bh * kCandRanges;
    } else {
        rg.base = w.surv + (int64_t)bh * a.row_stride;
        rg.stride = kFilterRows;
        rg.nreg = (int)((a.len + kFilterRows - 1) / kFilterRows);
        cnts = w.surv_cnt + (int64_t)bh * a.n_regions;
    }
    {
        // prefix over region counts: thread t owns regions [t*rpt, ...)
        const int rpt = (rg.nreg + NT - 1) / NT;
        const int r0 = tid * rpt < rg.nreg ? tid * rpt : rg.nreg;
        const int r1 = r0 + rpt < rg.nreg ? r0 + rpt : rg.nreg;
        uint32_t mine = 0;
        for (int r = r0; r < r1; ++r) mine += cnts[r];
        uint32_t total;
        uint32_t run = block_excl_scan<NT>(mine, sm.redu, &total);
        for (int r = r0; r < r1; ++r) {
            sm.pref[r] = run;
            run += cnts[r];
        }
        if (tid == 0) sm.pref[rg.nreg] = total;
        __syncthreads();
        rg.n = (int)total;
    }
    rg.pref = sm.pref;
    rg.staged = nullptr;
    if (rg.n <= kEntCache) {
        for (int j = tid; j < rg.n; j += NT) sm.ent[j] = rg.get(j);
        __syncthreads();
        rg.staged = sm.ent;
    }

    // Top-K (Eq. 1 / Eq. 11), then the selected entries in index order.
    uint64_t prefix, mask;
    radix_threshold<D, NT>(rg, a.K, sm, prefix, mask);
    const int kn = rg.n < a.K ? rg.n : a.K;
    {
        const int ept = (rg.n + NT - 1) / NT;
        const int j0 = tid * ept < rg.n ? tid * ept : rg.n;
        const int j1 = j0 + ept < rg.n ? j0 + ept : rg.n;
        uint32_t mine = 0;
        for (int j = j0; j < j1; ++j) mine += ((rg.get(j) & mask) >= prefix) ? 1u : 0u;
        uint32_t total;
        uint32_t pos = block_excl_scan<NT>(mine, sm.redu, &total);
        for (int j = j0; j < j1; ++j) {
            const uint64_t e = rg.get(j);
            if ((e & mask) >= prefix && pos < (uint32_t)kMaxK)
                sm.sel[pos++] = ((uint64_t)rank_index(e) << 32) | rank_key(e);
        }
        __syncthreads();
    }

    if (writes_out) {
        // Eq. 12 on this block's slice of the head dimension.
        float mx = -INFINITY;
        for (int t = tid; t < kn; t += NT) mx = fmaxf(mx, key_score((uint32_t)sm.sel[t]));
        mx = block_reduce<NT>(mx, sm.red32, [](float x, float y) { return fmaxf(x, y); });
        float lsum = 0.0f;
        for (int t = tid; t < kn; t += NT) {
            const float wt = expf(key_score((uint32_t)sm.sel[t]) - mx);
            sm.wgt[t] = wt;
            lsum += wt;
        }
        lsum = block_reduce<NT>(lsum, sm.red32, [](float x, float y) { return x + y; });
        const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;
        const T *vbase = (const T *)a.v + ((int64_t)b * a.Hkv + g) * a.max_len * D + slice * DS;
        const int sub = lane / LPR, vl = lane % LPR;
        float acc[EPV];
#pragma unroll
        for (int e = 0; e < EPV; ++e) acc[e] = 0.0f;
#pragma unroll 4
        for (int t = wave * RPW + sub; t < kn; t += NW * RPW) {
            const uint32_t idx = (uint32_t)(sm.sel[t] >> 32);
            const uint4 raw = ((const uint4 *)(vbase + (int64_t)idx * D))[vl];
            Dot<T>::axpy(raw, sm.wgt[t], acc);
        }
#pragma unroll
        for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
            for (int e = 0; e < EPV; ++e) acc[e] += __shfl_xor(acc[e], o);
        if (sub == 0)
#pragma unroll
            for (int e = 0; e < EPV; ++e) sm.part[wave][vl * EPV + e] = acc[e];
        __syncthreads();
        if (tid < DS) {
            float o = 0.0f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) o += sm.part[ww][tid];
            a.out[(int64_t)bh * D + slice * DS + tid] = kn > 0 ? o / lsum : 0.0f;
        }
    }
    if (slice != 0) return;

    if (writes_out && a.sel != nullptr)
        for (int t = tid; t < a.K; t += NT)
            a.sel[(int64_t)bh * a.K + t] = t < kn ? (int32_t)(sm.sel[t] >> 32) : -1;
    if (a.do_insert) {
        // Sec. 3.4: insert (q_bar, support) after either path.
        const int64_t e = (int64_t)bh * a.M + a.insert_slot;
        if (a.mode == MODE_SELECT) {
            for (int t = tid; t < D; t += NT) w.qbar[e * D + t] = w.qbar_cur[(int64_t)bh * D + t];
        } else {
            const T *q = (const T *)a.q + (int64_t)bh * a.q_head_stride;
            block_qbar<T, D, NT>(q, sm.qbar, sm.red64);
            for (int t = tid; t < D; t += NT) w.qbar[e * D + t] = sm.qbar[t];
        }
        for (int t = tid; t < a.K; t += NT)
            w.supp[e * a.K + t] = t < kn ? (int32_t)(sm.sel[t] >> 32) : -1;
        if (tid == 0) w.cnt[e] = kn;
    }
    if (reuse) {
        if (tid == 0) {
            atomicAdd(&w.stats[STAT_CAND_SUM], (unsigned long long)rg.n);
            atomicMax(&w.stats[STAT_CAND_MAX], (unsigned long long)rg.n);
        }
    } else {
        // leave the histogram zeroed for the next launch
        for (int i = tid; i < kHistBins; i += NT) w.hist[(int64_t)bh * kHistBins + i] = 0u;
    }
    if (a.dbg_ncand && tid == 0) a.dbg_ncand[bh] = reuse ? rg.n : 0;
    if (a.dbg_cand)
        for (int j = tid; j < a.cand_cap; j += NT)
            a.dbg_cand[(int64_t)bh * a.cand_cap + j] = (reuse && j < rg.n) ? (int32_t)rank_index(rg.get(j)) : -1;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

// Launch on stream s; with a start/stop event pair the events are attached to the
// dispatch itself, so they time exactly this kernel.
template <typename F, typename... Args>
static hipError_t launch(F kernel, dim3 grid, dim3 block, hipStream_t s, const Timing &tm,
                         Args... args)
{
    if (tm.start != nullptr)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, s, tm.start, tm.stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
    return hipGetLastError();
}

bool shape_supported(int dtype, int d, int g)
{
    return (dtype == 0 || dtype == 1) && (d == 64 || d == 128) &&
           (g == 1 || g == 2 || g == 4 || g == 8);
}

template <typename T, int D>
static hipError_t sim_impl(const StepArgs &a, const Ws &w, hipStream_t s, const Timing &tm)
{
    const int nsb = (a.M + kSimSlots - 1) / kSimSlots;
    return launch(k_sim<T, D>, dim3((unsigned)(a.B * a.Hq * nsb)), dim3(kSimThreads), s, tm, a, w);
}

template <typename T, int D, int G>
static hipError_t score_impl(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s,
                             const Timing &tm)
{
    const int blocks = geo.scan_blocks + geo.cand_blocks;
    return launch(k_score<T, D, G>, dim3((unsigned)blocks), dim3(kScoreThreads), s, tm, a, w, geo);
}

template <typename T, int D>
static hipError_t final_impl(const StepArgs &a, const Ws &w, hipStream_t s, const Timing &tm)
{
    return launch(k_final<T, D>, dim3((unsigned)(a.B * a.Hq * kFinalSlices)), dim3(kFinalThreads),
                  s, tm, a, w);
}

template <typename T, int D>
static hipError_t score_g(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s,
                          const Timing &tm)
{
    switch (a.G) {
    case 1: return score_impl<T, D, 1>(a, w, geo, s, tm);
    case 2: return score_impl<T, D, 2>(a, w, geo, s, tm);
    case 4: return score_impl<T, D, 4>(a, w, geo, s, tm);
    default: return score_impl<T, D, 8>(a, w, geo, s, tm);
    }
}

hipError_t launch_sim(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                      hipStream_t s, const Timing &tm)
{
    (void)geo;
    if (dtype == 1)
        return a.D == 64 ? sim_impl<uint16_t, 64>(a, w, s, tm) : sim_impl<uint16_t, 128>(a, w, s, tm);
    return a.D == 64 ? sim_impl<float, 64>(a, w, s, tm) : sim_impl<float, 128>(a, w, s, tm);
}
hipError_t launch_score(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                        hipStream_t s, const Timing &tm)
{
    if (dtype == 1)
        return a.D == 64 ? score_g<uint16_t, 64>(a, w, geo, s, tm) : score_g<uint16_t, 128>(a, w, geo, s, tm);
    return a.D == 64 ? score_g<float, 64>(a, w, geo, s, tm) : score_g<float, 128>(a, w, geo, s, tm);
}
hipError_t launch_filter(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                         hipStream_t s, const Timing &tm)
{
    (void)dtype;
    return launch(k_filter, dim3((unsigned)(a.B * a.Hq * geo.filter_blocks_per_head)),
                  dim3(kScoreThreads), s, tm, a, w, geo);
}
hipError_t launch_final(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                        hipStream_t s, const Timing &tm)
{
    (void)geo;
    if (dtype == 1)
        return a.D == 64 ? final_impl<uint16_t, 64>(a, w, s, tm) : final_impl<uint16_t, 128>(a, w, s, tm);
    return a.D == 64 ? final_impl<float, 64>(a, w, s, tm) : final_impl<float, 128>(a, w, s, tm);
}

}  // namespace retopk
