// retopk_kernels.hip -- gfx950 (CDNA4) kernels of the ReTopK decode step.
//
// One decode step is four launches on the caller's stream:
//   k_select  one block per query head: q_bar, cosine similarity to the cached
//             queries (Eq. 6), rho_max, Top-R (Eq. 7), the path rule (Eq. 13) and,
//             on reuse, the candidate set of Eq. 8-9 (union through an LDS bitmap,
//             emitted in ascending order).
//   k_score   full-history QK scan of every KV group that has an exact head
//             (Eq. 4; one key row load serves the G query heads of the group) with
//             a per-head score histogram, plus gathered QK on the candidate sets
//             of reuse heads (Eq. 10).
//   k_filter  for every exact head: keep the scores at or above the histogram bin
//             that holds the K-th largest.
//   k_final   one block per query head: Top-K over the head's candidates (Eq. 11)
//             or surviving scores (Eq. 1), Softmax-V (Eq. 12), outputs, and the
//             cache insert of Sec. 3.4.
// Exact Top-K attention alone is k_score (scan only) + k_filter + k_final.
// Blocks never wait on each other inside a launch: every hand-over between
// blocks goes through a kernel boundary.
//
// Ranking is on the fp32 scaled score fl32(q.k) * fl32(1/sqrt d) with ties to the
// lower index: every candidate carries a 64-bit rank (score key << 32 | ~index)
// and selection is a radix select over those distinct ranks.
#include "retopk_internal.h"

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

template <int G>
__device__ __forceinline__ float pick(const float (&acc)[G], int j)
{
    float r = acc[0];
#pragma unroll
    for (int t = 1; t < G; ++t)
        if (t == j) r = acc[t];
    return r;
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
// Final stage of one head: Top-K over rank entries, Softmax-V, outputs, insert.
// ---------------------------------------------------------------------------

template <int D, int NT>
struct FinalSmem {
    uint64_t ent[kEntCache];  // the head's entries, when they fit
    uint64_t sel[kMaxK];      // selected (index << 32 | score key), sorted by index
    float wgt[kMaxK];
    float part[NT / 64][D];
    uint32_t hist[256];
    float qbar[D];
    double red64[NT / 64];
    float red32[NT / 64];
    uint32_t found_digit, found_above, found_cnt, count;
};

// Selects the top min(K, n) of src[0..n) (distinct 64-bit ranks, larger is
// better), then sorts them by index.  Returns the number selected.
template <int D, int NT>
__device__ int select_topk(const uint64_t *src, int n, int K, FinalSmem<D, NT> &sm)
{
    const int tid = threadIdx.x;
    uint64_t prefix = 0, mask = 0;
    const bool all = n <= K;
    if (!all) {
        uint32_t k_rem = (uint32_t)K;
        // Radix select on 8-bit digits, most significant first: after each pass the
        // selected set is {rank : (rank & mask) > prefix} plus k_rem entries that
        // still match prefix under mask.
        for (int shift = 56; shift >= 0; shift -= 8) {
            for (int i = tid; i < 256; i += NT) sm.hist[i] = 0;
            __syncthreads();
            for (int i = tid; i < n; i += NT) {
                uint64_t e = src[i];
                if ((e & mask) == prefix) atomicAdd(&sm.hist[(e >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (tid < 64) {
                // lane l covers digits 255-4l, 254-4l, 253-4l, 252-4l (descending)
                uint32_t c[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) c[j] = sm.hist[255 - 4 * tid - j];
                uint32_t tot = c[0] + c[1] + c[2] + c[3];
                uint32_t above = wave_incl_scan(tot) - tot;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (above < k_rem && above + c[j] >= k_rem) {
                        sm.found_digit = 255u - 4u * tid - j;
                        sm.found_above = above;
                        sm.found_cnt = c[j];
                    }
                    above += c[j];
                }
            }
            __syncthreads();
            const uint32_t dgt = sm.found_digit;
            k_rem -= sm.found_above;
            prefix |= (uint64_t)dgt << shift;
            mask |= (uint64_t)0xFFu << shift;
            const bool done = sm.found_cnt == k_rem;
            __syncthreads();
            if (done) break;
        }
    }
    const int kn = all ? n : K;
    if (tid == 0) sm.count = 0;
    __syncthreads();
    for (int i = tid; i < n; i += NT) {
        uint64_t e = src[i];
        if (all || (e & mask) >= prefix) {
            uint32_t pos = atomicAdd(&sm.count, 1u);
            if (pos < (uint32_t)kMaxK) sm.sel[pos] = ((uint64_t)rank_index(e) << 32) | rank_key(e);
        }
    }
    int kp = 1;
    while (kp < kn) kp <<= 1;
    __syncthreads();
    for (int i = kn + tid; i < kp; i += NT) sm.sel[i] = ~0ull;
    __syncthreads();
    // Bitonic sort (ascending) of sel[0..kp) -> ascending index order.
    for (int k2 = 2; k2 <= kp; k2 <<= 1) {
        for (int j = k2 >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < kp; i += NT) {
                int ixj = i ^ j;
                if (ixj > i) {
                    uint64_t x = sm.sel[i], y = sm.sel[ixj];
                    bool up = (i & k2) == 0;
                    if ((x > y) == up) {
                        sm.sel[i] = y;
                        sm.sel[ixj] = x;
                    }
                }
            }
            __syncthreads();
        }
    }
    return kn;
}

// Top-K of ents[0..n), Softmax-V over the selected rows (Eq. 12), sel output and
// cache insert.
template <typename T, int D, int NT>
__device__ void finalize_head(const StepArgs &a, const Ws &w, int bh, const uint64_t *ents,
                              int n, FinalSmem<D, NT> &sm)
{
    using R = RowT<T, D>;
    constexpr int LPR = R::kBytes / 16;   // lanes per row for 16-byte loads
    constexpr int RPW = 64 / LPR;         // rows per wave instruction
    constexpr int EPV = R::kEPV;
    constexpr int NW = NT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;

    const uint64_t *src = ents;
    if (n <= kEntCache) {
        for (int i = tid; i < n; i += NT) sm.ent[i] = ents[i];
        __syncthreads();
        src = sm.ent;
    }
    const int kn = select_topk<D, NT>(src, n, a.K, sm);

    if (a.out != nullptr && a.mode != MODE_PREFILL) {
        float mx = -INFINITY;
        for (int t = tid; t < kn; t += NT) mx = fmaxf(mx, key_score((uint32_t)sm.sel[t]));
        mx = block_reduce<NT>(mx, sm.red32, [](float x, float y) { return fmaxf(x, y); });
        float lsum = 0.0f;
        for (int t = tid; t < kn; t += NT) {
            float wt = expf(key_score((uint32_t)sm.sel[t]) - mx);
            sm.wgt[t] = wt;
            lsum += wt;
        }
        lsum = block_reduce<NT>(lsum, sm.red32, [](float x, float y) { return x + y; });
        // block_reduce ends with a barrier, so wgt[] is visible here.
        const T *vbase = (const T *)a.v + ((int64_t)b * a.Hkv + g) * a.max_len * D;
        const int sub = lane / LPR, vl = lane % LPR;
        float acc[EPV];
#pragma unroll
        for (int e = 0; e < EPV; ++e) acc[e] = 0.0f;
#pragma unroll 8
        for (int t = wave * RPW + sub; t < kn; t += NW * RPW) {
            uint32_t idx = (uint32_t)(sm.sel[t] >> 32);
            uint4 raw = ((const uint4 *)(vbase + (int64_t)idx * D))[vl];
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
        if (tid < D) {
            float o = 0.0f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) o += sm.part[ww][tid];
            a.out[(int64_t)bh * D + tid] = kn > 0 ? o / lsum : 0.0f;
        }
    }
    if (a.sel != nullptr && a.mode != MODE_PREFILL) {
        for (int t = tid; t < a.K; t += NT)
            a.sel[(int64_t)bh * a.K + t] = t < kn ? (int32_t)(sm.sel[t] >> 32) : -1;
    }
    if (a.do_insert) {
        const T *q = (const T *)a.q + (int64_t)bh * a.q_head_stride;
        block_qbar<T, D, NT>(q, sm.qbar, sm.red64);
        const int64_t e = (int64_t)bh * a.M + a.insert_slot;
        for (int t = tid; t < D; t += NT) w.qbar[e * D + t] = sm.qbar[t];
        for (int t = tid; t < a.K; t += NT)
            w.supp[e * a.K + t] = t < kn ? (int32_t)(sm.sel[t] >> 32) : -1;
        if (tid == 0) w.cnt[e] = kn;
    }
}

// ---------------------------------------------------------------------------
// k_select: one block per query head
// ---------------------------------------------------------------------------

template <int D>
struct SelectSmem {
    uint32_t bitmap[kBitmapWords];
    double rho[kMaxCache];
    float qbar[D];
    double red64[kSelectThreads / 64];
    uint32_t red32[kSelectThreads / 64];
    double best_rho[kSelectThreads / 64];
    int32_t best_age[kSelectThreads / 64];
    int32_t best_slot[kSelectThreads / 64];
    int32_t ret[kMaxR];
    uint8_t taken[kMaxCache];
};

__device__ __forceinline__ bool better(double ra, int aa, double rb, int ab)
{
    return ra > rb || (ra == rb && aa < ab);
}

template <typename T, int D>
__global__ __launch_bounds__(kSelectThreads) void k_select(StepArgs a, Ws w, Geometry geo)
{
    constexpr int NT = kSelectThreads;
    constexpr int NW = NT / 64;
    __shared__ SelectSmem<D> sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.x;
    const int M = a.M;
    const int n_valid = (int)(a.n_ins < (int64_t)M ? a.n_ins : (int64_t)M);
    const T *q = (const T *)a.q + (int64_t)bh * a.q_head_stride;

    block_qbar<T, D, NT>(q, sm.qbar, sm.red64);

    // Eq. 6: 16 slots per wave pass, 4 lanes per cached row.
    {
        const int p = lane & 3;
        const float4 *cache = (const float4 *)(w.qbar + (int64_t)bh * M * D);
        for (int base = 0; base < n_valid; base += NW * 16) {
            const int slot = base + wave * 16 + (lane >> 2);
            float4 c[D / 16];
#pragma unroll
            for (int s = 0; s < D / 16; ++s)
                c[s] = slot < n_valid ? cache[(int64_t)slot * (D / 4) + s * 4 + p]
                                      : make_float4(0.f, 0.f, 0.f, 0.f);
            double acc = 0.0;
#pragma unroll
            for (int s = 0; s < D / 16; ++s) {
                const float *qq = &sm.qbar[(s * 4 + p) * 4];
                acc += (double)c[s].x * (double)qq[0];
                acc += (double)c[s].y * (double)qq[1];
                acc += (double)c[s].z * (double)qq[2];
                acc += (double)c[s].w * (double)qq[3];
            }
            acc = quad_sum(acc);
            if (slot < n_valid && p == 0) sm.rho[slot] = acc;
        }
    }
    __syncthreads();

    double mx = -INFINITY;
    for (int i = tid; i < n_valid; i += NT) mx = fmax(mx, sm.rho[i]);
    mx = block_reduce<NT>(mx, sm.red64, [](double x, double y) { return fmax(x, y); });

    // Eq. 13 (no refresh in this mode): exact path iff rho_max < tau.
    const int8_t path = mx < (double)a.tau ? PATH_FALLBACK : PATH_REUSE;
    if (tid == 0) {
        w.path[bh] = path;
        if (a.dbg_path) a.dbg_path[bh] = path;
        if (a.dbg_rho) a.dbg_rho[bh] = mx;
        atomicAdd(&w.stats[path == PATH_REUSE ? STAT_REUSE : STAT_FALLBACK], 1ull);
    }
    const int nret = path == PATH_REUSE ? (a.R < n_valid ? a.R : n_valid) : 0;

    // Eq. 7: the nret most similar slots; equal similarity -> newer insertion
    // (smaller age = (n_ins - 1 - slot) mod C).
    for (int i = tid; i < n_valid; i += NT) sm.taken[i] = 0;
    __syncthreads();
    for (int r = 0; r < nret; ++r) {
        double br = -INFINITY;
        int ba = 0x7FFFFFFF, bs = -1;
        for (int i = tid; i < n_valid; i += NT) {
            if (sm.taken[i]) continue;
            int age = (int)(((a.n_ins - 1 - i) % M + M) % M);
            if (bs < 0 || better(sm.rho[i], age, br, ba)) { br = sm.rho[i]; ba = age; bs = i; }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            double orr = __shfl_xor(br, o);
            int oa = __shfl_xor(ba, o), os = __shfl_xor(bs, o);
            if (os >= 0 && (bs < 0 || better(orr, oa, br, ba))) { br = orr; ba = oa; bs = os; }
        }
        if (lane == 0) { sm.best_rho[wave] = br; sm.best_age[wave] = ba; sm.best_slot[wave] = bs; }
        __syncthreads();
        if (tid == 0) {
            double fr = sm.best_rho[0];
            int fa = sm.best_age[0], fs = sm.best_slot[0];
            for (int ww = 1; ww < NW; ++ww) {
                int os = sm.best_slot[ww];
                if (os >= 0 && (fs < 0 || better(sm.best_rho[ww], sm.best_age[ww], fr, fa))) {
                    fr = sm.best_rho[ww]; fa = sm.best_age[ww]; fs = os;
                }
            }
            sm.ret[r] = fs;
            sm.taken[fs] = 1;
        }
        __syncthreads();
    }
    if (a.dbg_ret)
        for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = i < nret ? sm.ret[i] : -1;

    int total = 0;
    if (path == PATH_REUSE) {
        // Eq. 8-9: union of the retrieved supports and the window [len-W, len),
        // through a bitmap over index segments; compaction emits ascending order.
        const int64_t len = a.len;
        const int64_t w0 = len - a.W > 0 ? len - a.W : 0;
        int32_t *cand = w.cand + (int64_t)bh * a.cand_cap;
        int32_t *dcand = a.dbg_cand ? a.dbg_cand + (int64_t)bh * a.cand_cap : nullptr;
        for (int64_t lo = 0; lo < len; lo += (int64_t)kBitmapWords * 32) {
            const int64_t hi = (lo + (int64_t)kBitmapWords * 32 < len) ? lo + (int64_t)kBitmapWords * 32 : len;
            const int nwords = (int)((hi - lo + 31) >> 5);
            for (int i = tid; i < nwords; i += NT) sm.bitmap[i] = 0u;
            __syncthreads();
            for (int r = 0; r < nret; ++r) {
                const int64_t e = (int64_t)bh * M + sm.ret[r];
                const int32_t *sp = w.supp + e * a.K;
                const int c = w.cnt[e];
                for (int t = tid; t < c; t += NT) {
                    int64_t x = sp[t];
                    if (x >= lo && x < hi) atomicOr(&sm.bitmap[(x - lo) >> 5], 1u << ((x - lo) & 31));
                }
            }
            for (int64_t x = (w0 > lo ? w0 : lo) + tid; x < hi; x += NT)
                atomicOr(&sm.bitmap[(x - lo) >> 5], 1u << ((x - lo) & 31));
            __syncthreads();
            const int wpt = (nwords + NT - 1) / NT;
            const int wb = tid * wpt;
            const int we = (wb + wpt < nwords) ? wb + wpt : nwords;
            uint32_t mine = 0;
            for (int i = wb; i < we; ++i) mine += __popc(sm.bitmap[i]);
            uint32_t seg_total;
            uint32_t pos = (uint32_t)total + block_excl_scan<NT>(mine, sm.red32, &seg_total);
            for (int i = wb; i < we; ++i) {
                uint32_t bits = sm.bitmap[i];
                while (bits) {
                    int bit = __ffs(bits) - 1;
                    bits &= bits - 1u;
                    int32_t x = (int32_t)(lo + (int64_t)i * 32 + bit);
                    cand[pos] = x;
                    if (dcand) dcand[pos] = x;
                    ++pos;
                }
            }
            total += (int)seg_total;
            __syncthreads();
        }
        if (tid == 0) {
            atomicAdd(&w.stats[STAT_CAND_SUM], (unsigned long long)total);
            atomicMax(&w.stats[STAT_CAND_MAX], (unsigned long long)total);
        }
    }
    if (tid == 0) {
        w.n_cand[bh] = total;
        if (a.dbg_ncand) a.dbg_ncand[bh] = total;
    }
    if (a.dbg_cand)
        for (int i = total + tid; i < a.cand_cap; i += NT) a.dbg_cand[(int64_t)bh * a.cand_cap + i] = -1;
}

// ---------------------------------------------------------------------------
// k_score: full-history scan blocks, then candidate blocks
// ---------------------------------------------------------------------------

template <typename T, int D, int G>
__device__ void scan_block(const StepArgs &a, const Ws &w, const Geometry &geo, uint32_t *s_hist)
{
    using R = RowT<T, D>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int chunks = geo.scan_blocks / (a.B * a.Hkv);
    const int bg = blockIdx.x / chunks, chunk = blockIdx.x % chunks;
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    const int bh0 = b * a.Hq + g * G;

    uint32_t exmask = 0;
#pragma unroll
    for (int j = 0; j < G; ++j) {
        bool ex = a.mode != MODE_SELECT || w.path[bh0 + j] != PATH_REUSE;
        exmask |= (uint32_t)ex << j;
    }
    if (exmask == 0) return;
    const int64_t row0 = (int64_t)chunk * geo.scan_chunk_rows;
    if (row0 >= a.len) return;
    if (a.mode == MODE_SELECT && chunk == 0 && tid == 0) atomicAdd(&w.stats[STAT_SCANS], 1ull);

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
                acc[j] = quad_sum(s0);
            }
            if (row[u] < row_end) {
#pragma unroll
                for (int jj = 0; jj < (G + 3) / 4; ++jj) {
                    const int j = jj * 4 + p;
                    if (j < G && ((exmask >> j) & 1u)) {
                        const float sc = pick<G>(acc, j) * a.inv_sqrt_d;
                        w.scores[(int64_t)(bh0 + j) * a.max_len + row[u]] = sc;
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

template <typename T, int D>
__device__ void cand_block(const StepArgs &a, const Ws &w, const Geometry &geo, int cb)
{
    using R = RowT<T, D>;
    constexpr int kIters = kCandRows / kScanRowsPerIter;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int bh = cb / geo.cand_blocks_per_head, cc = cb % geo.cand_blocks_per_head;
    if (w.path[bh] != PATH_REUSE) return;
    const int n = w.n_cand[bh];
    if (cc * kCandRows >= n) return;
    const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;

    uint4 qv[R::kNV];
    const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)bh * a.q_head_stride);
#pragma unroll
    for (int s = 0; s < R::kNV; ++s) qv[s] = qr[s * 4 + p];
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    const int32_t *cl = w.cand + (int64_t)bh * a.cand_cap;
    uint64_t *ce = w.cand_ent + (int64_t)bh * a.cand_cap;

    uint4 kv[kIters][R::kNV];
    int ci[kIters], cidx[kIters];
#pragma unroll
    for (int u = 0; u < kIters; ++u) {
        ci[u] = cc * kCandRows + u * kScanRowsPerIter + wave * 16 + rl;
        cidx[u] = ci[u] < n ? cl[ci[u]] : 0;
        if (ci[u] < n) {
            const uint4 *rp = (const uint4 *)(kbase + (int64_t)cidx[u] * D);
#pragma unroll
            for (int s = 0; s < R::kNV; ++s) kv[u][s] = rp[s * 4 + p];
        } else {
#pragma unroll
            for (int s = 0; s < R::kNV; ++s) kv[u][s] = make_uint4(0u, 0u, 0u, 0u);
        }
    }
#pragma unroll
    for (int u = 0; u < kIters; ++u) {
        float s0 = 0.0f;
#pragma unroll
        for (int s = 0; s < R::kNV; ++s) s0 = Dot<T>::f(kv[u][s], qv[s], s0);
        s0 = quad_sum(s0);
        if (p == 0 && ci[u] < n) ce[ci[u]] = rank_of(s0 * a.inv_sqrt_d, (uint32_t)cidx[u]);
    }
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kScoreThreads) void k_score(StepArgs a, Ws w, Geometry geo)
{
    __shared__ uint32_t s_hist[G * kHistBins];
    if ((int)blockIdx.x < geo.scan_blocks)
        scan_block<T, D, G>(a, w, geo, s_hist);
    else
        cand_block<T, D>(a, w, geo, (int)blockIdx.x - geo.scan_blocks);
}

// ---------------------------------------------------------------------------
// k_filter: the surviving scores of every exact head
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kScoreThreads) void k_filter(StepArgs a, Ws w, Geometry geo)
{
    constexpr int NT = kScoreThreads;
    static_assert(NT * 4 == kHistBins, "4 histogram bins per thread");
    __shared__ uint32_t s_red[NT / 64];
    __shared__ uint32_t s_bstar;
    const int tid = threadIdx.x;
    const int bh = blockIdx.x / geo.filter_blocks_per_head;
    const int fc = blockIdx.x % geo.filter_blocks_per_head;
    if (a.mode == MODE_SELECT && w.path[bh] == PATH_REUSE) return;

    // The bin b* that holds the kn-th largest score: the largest b with
    // count(bins >= b) >= kn.  Thread t holds bins 2047-4t .. 2044-4t.
    {
        const uint32_t kn = (uint32_t)(a.K < a.len ? a.K : a.len);
        const uint32_t *hist = w.hist + (int64_t)bh * kHistBins;
        uint32_t c[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) c[j] = hist[kHistBins - 1 - 4 * tid - j];
        uint32_t tot = c[0] + c[1] + c[2] + c[3], all;
        uint32_t above = block_excl_scan<NT>(tot, s_red, &all);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (above < kn && above + c[j] >= kn) s_bstar = (uint32_t)(kHistBins - 1 - 4 * tid - j);
            above += c[j];
        }
        __syncthreads();
    }
    const uint32_t kmin = s_bstar << kHistShift;
    const float *sc = w.scores + (int64_t)bh * a.max_len;
    uint64_t *sv = w.surv + (int64_t)bh * a.max_len;
    const int64_t i0 = (int64_t)fc * kFilterRows;
    float s[kFilterRows / NT];
#pragma unroll
    for (int it = 0; it < kFilterRows / NT; ++it) {
        const int64_t i = i0 + (int64_t)it * NT + tid;
        s[it] = i < a.len ? sc[i] : 0.0f;
    }
#pragma unroll
    for (int it = 0; it < kFilterRows / NT; ++it) {
        const int64_t i = i0 + (int64_t)it * NT + tid;
        const bool keep = i < a.len && ord_key(s[it]) >= kmin;
        const uint64_t m = __ballot(keep);
        if (m) {
            const int lane = tid & 63;
            const int leader = __ffsll((unsigned long long)m) - 1;
            uint32_t base = 0;
            if (lane == leader) base = atomicAdd(&w.surv_count[bh], (uint32_t)__popcll(m));
            base = __shfl(base, leader);
            const uint32_t off = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
            if (keep) sv[base + off] = rank_of(s[it], (uint32_t)i);
        }
    }
}

// ---------------------------------------------------------------------------
// k_final: one block per query head
// ---------------------------------------------------------------------------

template <typename T, int D>
__global__ __launch_bounds__(kFinalThreads) void k_final(StepArgs a, Ws w, Geometry geo)
{
    constexpr int NT = kFinalThreads;
    __shared__ FinalSmem<D, NT> sm;
    const int tid = threadIdx.x;
    const int bh = blockIdx.x;
    (void)geo;

    if (a.mode == MODE_REFRESH || a.mode == MODE_COLD) {
        const int8_t code = a.mode == MODE_REFRESH ? PATH_REFRESH : PATH_COLD;
        if (tid == 0) {
            if (a.dbg_path) a.dbg_path[bh] = code;
            if (a.dbg_rho) a.dbg_rho[bh] = __builtin_nan("");
            if (a.dbg_ncand) a.dbg_ncand[bh] = 0;
        }
        if (a.dbg_ret)
            for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = -1;
        if (a.dbg_cand)
            for (int i = tid; i < a.cand_cap; i += NT) a.dbg_cand[(int64_t)bh * a.cand_cap + i] = -1;
    }
    const bool reuse = a.mode == MODE_SELECT && w.path[bh] == PATH_REUSE;
    if (reuse) {
        finalize_head<T, D, NT>(a, w, bh, w.cand_ent + (int64_t)bh * a.cand_cap, w.n_cand[bh], sm);
    } else {
        const int n = (int)w.surv_count[bh];
        finalize_head<T, D, NT>(a, w, bh, w.surv + (int64_t)bh * a.max_len, n, sm);
        // Leave the exact-path workspace zeroed for the next launch.
        for (int i = tid; i < kHistBins; i += NT) w.hist[(int64_t)bh * kHistBins + i] = 0u;
        if (tid == 0) w.surv_count[bh] = 0u;
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

bool shape_supported(int dtype, int d, int g)
{
    return (dtype == 0 || dtype == 1) && (d == 64 || d == 128) &&
           (g == 1 || g == 2 || g == 4 || g == 8);
}

template <typename T, int D>
static hipError_t select_impl(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    hipLaunchKernelGGL((k_select<T, D>), dim3((unsigned)(a.B * a.Hq)), dim3(kSelectThreads), 0, s,
                       a, w, geo);
    return hipGetLastError();
}

template <typename T, int D, int G>
static hipError_t score_impl(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    const int blocks = geo.scan_blocks + a.B * a.Hq * geo.cand_blocks_per_head;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((k_score<T, D, G>), dim3((unsigned)blocks), dim3(kScoreThreads), 0, s, a, w, geo);
    return hipGetLastError();
}

static hipError_t filter_impl(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    dim3 grid((unsigned)(a.B * a.Hq * geo.filter_blocks_per_head));
    hipLaunchKernelGGL(k_filter, grid, dim3(kScoreThreads), 0, s, a, w, geo);
    return hipGetLastError();
}

template <typename T, int D>
static hipError_t final_impl(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    hipLaunchKernelGGL((k_final<T, D>), dim3((unsigned)(a.B * a.Hq)), dim3(kFinalThreads), 0, s,
                       a, w, geo);
    return hipGetLastError();
}

template <typename T>
static hipError_t select_d(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    return a.D == 64 ? select_impl<T, 64>(a, w, geo, s) : select_impl<T, 128>(a, w, geo, s);
}
template <typename T>
static hipError_t final_d(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    return a.D == 64 ? final_impl<T, 64>(a, w, geo, s) : final_impl<T, 128>(a, w, geo, s);
}
template <typename T, int D>
static hipError_t score_g(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    switch (a.G) {
    case 1: return score_impl<T, D, 1>(a, w, geo, s);
    case 2: return score_impl<T, D, 2>(a, w, geo, s);
    case 4: return score_impl<T, D, 4>(a, w, geo, s);
    default: return score_impl<T, D, 8>(a, w, geo, s);
    }
}
template <typename T>
static hipError_t score_d(const StepArgs &a, const Ws &w, const Geometry &geo, hipStream_t s)
{
    return a.D == 64 ? score_g<T, 64>(a, w, geo, s) : score_g<T, 128>(a, w, geo, s);
}

hipError_t launch_select(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                         hipStream_t s)
{
    return dtype == 1 ? select_d<uint16_t>(a, w, geo, s) : select_d<float>(a, w, geo, s);
}
hipError_t launch_score(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                        hipStream_t s)
{
    return dtype == 1 ? score_d<uint16_t>(a, w, geo, s) : score_d<float>(a, w, geo, s);
}
hipError_t launch_filter(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                         hipStream_t s)
{
    (void)dtype;
    return filter_impl(a, w, geo, s);
}
hipError_t launch_final(int dtype, const StepArgs &a, const Ws &w, const Geometry &geo,
                        hipStream_t s)
{
    return dtype == 1 ? final_d<uint16_t>(a, w, geo, s) : final_d<float>(a, w, geo, s);
}

}  // namespace retopk
