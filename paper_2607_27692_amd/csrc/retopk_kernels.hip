// retopk_kernels.hip -- gfx950 (CDNA4) kernels of the ReTopK decode step.
//
// One decode step is four launches on the caller's stream, and blocks never wait
// on each other inside a launch (every hand-over is a kernel boundary):
//   k_sim     cosine similarity of q_bar to every cached query (Eq. 5, Eq. 6),
//             64 cache slots per block: each block's Top-R list, and a per-head
//             flag set when some block's best similarity reaches tau.
//   k_score   (a) full-history QK scan of every KV group with an exact head
//             (Eq. 4): one key-row load serves the G query heads of the group, and
//             each block adds its scores to a per-head histogram;
//             (b) for every query head, kCandRanges blocks each own one index range:
//             they apply the path rule (Eq. 13), take the Top-R cache entries
//             (Eq. 7), form the range's part of the candidate set (Eq. 8-9) through
//             an LDS bitmap and score those keys (Eq. 10).
//   k_filter  per exact head, the scores at or above the histogram bin that holds
//             the K-th largest, compacted in index order.
//   k_final   2, 4 or 8 blocks per head: each selects the Top-K of the head's
//             candidates (Eq. 11) or surviving scores (Eq. 1) -- entries held in
//             registers, value-linear score bins, the threshold bin ranked exactly
//             (a radix select on 64-bit ranks for the heads that do not fit) --
//             then aggregates one slice of the head dimension of Softmax-V
//             (Eq. 12); the writes of the support and of the cache entry
//             (Sec. 3.4) are shared out over the slices.
// Exact Top-K attention alone is the full-history scan (k_scan_list where every
// CU can own one whole 4096-row filter region, keeping each region's scores in
// LDS and writing its local survivors; otherwise k_score's scan blocks) +
// k_filter + k_final.
// A head's similarity, range and final blocks run on one XCD (blocks are placed
// on XCDs round-robin by block index), so that blocks sharing a head's data
// (Top-R lists, supports, value rows) share that XCD's L2.
//
// Ranking is on the fp32 scaled score fl32(q.k) * fl32(1/sqrt d) with ties to the
// lower index: every entry carries a 64-bit rank (score key << 32 | ~index), and
// ranks are distinct.
#include "retopk_internal.h"

#include <hip/hip_ext.h>

namespace retopk {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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
constexpr int kHalfMirror = 0x141; // row_half_mirror: lane i <-> 7 - i in each 8 lanes

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

// Inclusive prefix sum over the 64 lanes of a wave: Hillis-Steele inside each row
// of 16 lanes (DPP row shifts, lanes shifted in from outside the row read 0), then
// the row totals carried across rows with the row broadcasts of lanes 15 and 31.
// Reductions over a wave: DPP inside each row of 16 lanes (quad swaps, half-row
// and row mirrors), then the four row results read as scalars.  Every lane gets
// the result.
__device__ __forceinline__ uint32_t row_max_u32(uint32_t x)
{
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, kQuadXor1, 0xF, 0xF, true));
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, kQuadXor2, 0xF, 0xF, true));
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, kHalfMirror, 0xF, 0xF, true));
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, true));   // row_mirror
    return x;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x)
{
    x = row_max_u32(x);
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 0);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 16);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 32);
    const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)x, 48);
    return max(max(r0, r1), max(r2, r3));
}
__device__ __forceinline__ float wave_sum_f32(float x)
{
    x += dpp_f32<kQuadXor1>(x);
    x += dpp_f32<kQuadXor2>(x);
    x += dpp_f32<kHalfMirror>(x);
    x += dpp_f32<0x140>(x);   // row_mirror
    const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
    const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16));
    const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
    const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 48));
    return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ double wave_max_f64(double x)
{
    x = fmax(x, dpp_f64<kQuadXor1>(x));
    x = fmax(x, dpp_f64<kQuadXor2>(x));
    x = fmax(x, dpp_f64<kHalfMirror>(x));
    x = fmax(x, dpp_f64<0x140>(x));   // row_mirror
    auto rl = [&](int l) {
        const uint64_t u = __builtin_bit_cast(uint64_t, x);
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
        return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
    };
    return fmax(fmax(rl(0), rl(16)), fmax(rl(32), rl(48)));
}

// x from lane (i + n) mod 16 of the same row of 16 lanes (DPP row_ror:n, 1..15).
__device__ __forceinline__ float row_ror_f32(float x, int n)
{
    int r;
    switch (n) {
    case 1: r = __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x121, 0xF, 0xF, true); break;
    case 2: r = __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x122, 0xF, 0xF, true); break;
    case 4: r = __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x124, 0xF, 0xF, true); break;
    default: r = __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x128, 0xF, 0xF, true); break;
    }
    return __builtin_bit_cast(float, r);
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x)
{
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return x;
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

// Waves per SIMD that k_score is built for: 4 (two 512-thread blocks per CU), or
// 2 (256 registers a lane) where the group's query vectors and the two key rows a
// lane holds in flight would take more than 96 of 128 registers (G + 2 rows of
// kNV * 4 in the quad layout), or, in the octet layout of the fp32 8-head build,
// where the query vectors alone would take half of them (the bf16 8-head build
// holds D / 32 MFMA operands).
template <typename T, int D, int G>
constexpr int kGroupWaves = (G == 8 && sizeof(T) == 2) ? 4
                            : G == 8 ? (2 * G * RowT<T, D>::kNV > 64 ? 2 : 4)
                                     : ((G + 2) * RowT<T, D>::kNV * 4 > 96 ? 2 : 4);
// The same for k_dense, whose lanes also hold G value accumulators of kEPV floats
// (the 8-head build takes its scores in the octet layout, its queries dead by
// the time the accumulators live).
template <typename T, int D, int G>
constexpr int kDenseWaves = G == 8 ? (16 * RowT<T, D>::kNV > 64 ? 2 : 4)
                                   : (G * (4 * RowT<T, D>::kNV + RowT<T, D>::kEPV) > 96 ? 2 : 4);

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

// Reduce-scatter inside an octet of lanes (8 lanes per row, one per head of an
// 8-head group): lane o holds partial sums of the 8 dot products and returns the
// full (8-lane) sum of dot product o.  Three butterfly steps, as in
// quad_transpose_sum; the first pairs lane o with lane 7 - o (a DPP half-row
// mirror), whose bit 2 is the opposite of o's, which is all the step needs.
__device__ __forceinline__ float octet_transpose_sum(const float (&acc)[8], int o)
{
    const bool b2 = (o & 4) != 0, b1 = (o & 2) != 0, b0 = (o & 1) != 0;
    float h4[4], h2[2];
#pragma unroll
    for (int i = 0; i < 4; ++i)   // heads (o & 4) + i
        h4[i] = (b2 ? acc[i + 4] : acc[i]) + dpp_f32<kHalfMirror>(b2 ? acc[i] : acc[i + 4]);
#pragma unroll
    for (int i = 0; i < 2; ++i)   // heads (o & 6) + i
        h2[i] = (b1 ? h4[i + 2] : h4[i]) + dpp_f32<kQuadXor2>(b1 ? h4[i] : h4[i + 2]);
    return (b0 ? h2[1] : h2[0]) + dpp_f32<kQuadXor1>(b0 ? h2[0] : h2[1]);   // head o
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

// Age of a cache slot: 0 for the most recent insertion, (n_ins - 1 - slot) mod C.
__device__ __forceinline__ int slot_age(int age0, int slot, int M)
{
    const int a = age0 - slot;
    return a < 0 ? a + M : a;
}

template <typename T, int D>
__global__ __launch_bounds__(kSimThreads) void k_sim(StepArgs a, Ws w)
{
    constexpr int NT = kSimThreads;
    __shared__ float s_qbar[D];
    __shared__ double s_red[NT / 64];
    __shared__ __attribute__((aligned(16))) double s_rho[kSimSlots];
    __shared__ __attribute__((aligned(16))) int s_age[kSimSlots];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3;
    const int M = a.M;
    const int nsb = (M + kSimSlots - 1) / kSimSlots;
    // the nsb blocks of head bh run on XCD bh % 8 (block j is placed on XCD j % 8),
    // with the head's range blocks and final blocks, which read what they write
    const int xcd = (int)blockIdx.x & 7, rest = (int)blockIdx.x >> 3;
    const int sb = rest % nsb, bh = (rest / nsb) * 8 + xcd;
    if (bh >= a.B * a.Hq) return;
    const int n_valid = (int)(a.n_ins < (int64_t)M ? a.n_ins : (int64_t)M);

    // Eq. 6: 16 slots per wave, 4 lanes per cached row of D floats.  The cached
    // rows are loaded first, so that their latency overlaps the normalisation.
    const int local = wave * 16 + (lane >> 2);
    const int slot = sb * kSimSlots + local;
    const float4 *crow = (const float4 *)(w.qbar + ((int64_t)bh * M + (slot < n_valid ? slot : 0)) * D);
    float4 c[D / 16];
#pragma unroll
    for (int s = 0; s < D / 16; ++s) c[s] = crow[s * 4 + p];   // clamped row: always in bounds
    const int scnt = w.cnt[(int64_t)bh * M + (slot < n_valid ? slot : 0)];

    block_qbar<T, D, NT>((const T *)a.q + (int64_t)bh * a.q_head_stride, s_qbar, s_red);
    if (sb == 0)
        for (int t = tid; t < D; t += NT) w.qbar_cur[(int64_t)bh * D + t] = s_qbar[t];

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
    const int age0 = a.insert_slot > 0 ? a.insert_slot - 1 : M - 1;   // slot of the newest entry
    if (p == 0) {
        s_rho[local] = slot < n_valid ? acc : -INFINITY;
        s_age[local] = slot < n_valid ? slot_age(age0, slot, M) : 0x7FFFFFFF;
    }
    __syncthreads();

    // This block's Top-R slots (Eq. 7) by rank counting: the 4 lanes of a quad
    // compare slot `local` against 16 slots each; rank = number of slots that are
    // more similar, or equally similar and newer (with recent-R retrieval: that
    // are newer).  The global Top-R is contained in the union of the blocks'
    // lists.  The head's reuse flag is set when the block's best similarity over
    // the entries retrieval can use reaches tau: every valid slot for Eq. 7, the R
    // most recent for recent-R.
    const bool recent = a.retrieval == 1;
    {
        const double ri = s_rho[local];
        const int ai = s_age[local];
        // the 16 slots this lane compares against, read (16-byte reads) before
        // any comparison, then counted without branches
        double ro[16];
        int ao[16];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const double2 x = ((const double2 *)&s_rho[p * 16])[u];
            ro[2 * u] = x.x;
            ro[2 * u + 1] = x.y;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int4 x = ((const int4 *)&s_age[p * 16])[u];
            ao[4 * u] = x.x;
            ao[4 * u + 1] = x.y;
            ao[4 * u + 2] = x.z;
            ao[4 * u + 3] = x.w;
        }
        int cnt = 0;
        if (recent) {
#pragma unroll
            for (int u = 0; u < 16; ++u) cnt += ao[u] < ai ? 1 : 0;
        } else {
#pragma unroll
            for (int u = 0; u < 16; ++u)
                cnt += ((ro[u] > ri) | ((ro[u] == ri) & (ao[u] < ai))) ? 1 : 0;
        }
        cnt += __builtin_amdgcn_mov_dpp(cnt, kQuadXor1, 0xF, 0xF, true);
        cnt += __builtin_amdgcn_mov_dpp(cnt, kQuadXor2, 0xF, 0xF, true);
        const int64_t base = ((int64_t)bh * (kMaxCache / kSimSlots) + sb) * kMaxR;
        const bool listed = slot < n_valid && cnt < a.R && (!recent || ai < a.R);
        if (p == 0 && listed) {
            w.topr[base + cnt] = slot;
            w.topr_rho[base + cnt] = ri;
            w.topr_cnt[base + cnt] = scnt;
            // the head reuses (Eq. 13) iff some block's best similarity is >= tau
            // (every such block stores the same flag)
            if (cnt == 0 && !recent && ri >= (double)a.tau) w.reuse[bh] = 1;
        }
    }
    if (recent && wave == 0) {
        // one lane per slot of the block; list positions past this block's
        // retrieved entries are marked empty
        static_assert(kSimSlots == 64, "one lane per slot");
        const bool ret = sb * kSimSlots + lane < n_valid && s_age[lane] < a.R;
        double m = ret ? s_rho[lane] : -INFINITY;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
        const int listed = __popcll(__ballot(ret));
        const int64_t base = ((int64_t)bh * (kMaxCache / kSimSlots) + sb) * kMaxR;
        if (lane >= listed && lane < a.R) {
            w.topr[base + lane] = -1;
            w.topr_rho[base + lane] = -INFINITY;
            w.topr_cnt[base + lane] = 0;
        }
        if (lane == 0 && m >= (double)a.tau) w.reuse[bh] = 1;
    }
}

// ---------------------------------------------------------------------------
// k_score
// ---------------------------------------------------------------------------

// Dynamic LDS of k_score (bytes): the scan blocks' histograms, or a range
// block's Top-R merge candidates (24 bytes each), which later hold the union
// bitmap segment and the candidate list.
__host__ __device__ constexpr int score_scan_lds(int g) { return g * kHistBins * 4; }
__host__ __device__ constexpr int score_range_lds(int n_merge)
{
    return 24 * n_merge > kSegWords * 4 + kCandList * 4 ? 24 * n_merge : kSegWords * 4 + kCandList * 4;
}
constexpr int kLocalGroups = 512;   // exact KV groups one scan block's rows can touch

// Adds a scan segment's per-head LDS histograms (G rows of kHistBins counts) to
// the global histograms of the group's exact heads (bits of exmask).
template <int G>
__device__ void flush_hist(const Ws &w, int bh0, uint32_t exmask, const uint32_t *s_hist)
{
    for (int i = threadIdx.x; i < G * kHistBins; i += kScoreThreads) {
        const int j = i / kHistBins;
        if ((exmask >> j) & 1u) {
            const uint32_t c = s_hist[i];
            if (c) atomicAdd(&w.hist[(int64_t)(bh0 + j) * kHistBins + (i % kHistBins)], c);
        }
    }
}

// scan_segment for the fp32 8-head build (groups of 5 to 8): a key row is split over
// the 8 lanes of an octet, lane o loading 16-byte vectors s * 8 + o, so that each
// lane holds half the query registers of the quad layout, and after the octet
// reduce-scatter lane o owns head o's score.  64 rows per pass of the block, 4
// passes (256 rows) per iteration, loaded from clamped (in-bounds) rows.
template <typename T, int D>
__device__ void scan_segment_octet(const StepArgs &a, const Ws &w, int b, int g, uint32_t exmask,
                                   int64_t row0, int64_t row1, uint32_t *s_hist)
{
    constexpr int G = 8;
    constexpr int NV = RowT<T, D>::kBytes / 128;          // vectors per lane per row
    constexpr int RPP = kScoreThreads / 8;                // rows per pass
    constexpr int UP = 2 * kScanRowsPerIter / RPP;        // passes per iteration
    static_assert(NV >= 1 && UP * RPP == 2 * kScanRowsPerIter, "octet row geometry");
    const int tid = threadIdx.x, o = tid & 7, rr = tid >> 3;
    const int bh0 = b * a.Hq + g * a.G;
    if (a.mode == MODE_SELECT && row0 == 0 && tid == 0) atomicAdd(&w.stats[STAT_SCANS], 1ull);
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    uint4 qv[G][NV];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const int hj = j < a.G ? j : 0;   // heads past a.G pad the group
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)(bh0 + hj) * a.q_head_stride);
#pragma unroll
        for (int s = 0; s < NV; ++s) qv[j][s] = qr[s * 8 + o];
    }
    // head o's scores are stored when it is exact, or (in a scan-fed step) when
    // it reuses in a scanned group, for its candidates; only exact heads are
    // counted in the histograms
    const bool keep = o < a.G && (((exmask >> o) & 1u) || a.scan_fed);
    const bool count = o < a.G && ((exmask >> o) & 1u);
    uint4 kv[UP][NV];
    int row[UP];                          // rows < len < 2^31
    auto load = [&](int64_t base) {
#pragma unroll
        for (int u = 0; u < UP; ++u) {
            row[u] = (int)base + u * RPP + rr;
            const uint4 *rp = (const uint4 *)(kbase + (row[u] < row1 ? (int64_t)row[u] : row0) * D);
#pragma unroll
            for (int s = 0; s < NV; ++s) kv[u][s] = rp[s * 8 + o];
        }
    };
    load(row0);   // the first rows are in flight while the histogram is cleared
    __syncthreads();   // the previous segment's histogram flush is done
    for (int i = tid; i < G * kHistBins; i += kScoreThreads) s_hist[i] = 0u;
    __syncthreads();

    for (int64_t base = row0; base < row1;) {
#pragma unroll
        for (int u = 0; u < UP; ++u) {
            float acc[G];
#pragma unroll
            for (int j = 0; j < G; ++j) {
                float s0 = 0.0f;
#pragma unroll
                for (int s = 0; s < NV; ++s) s0 = Dot<T>::f(kv[u][s], qv[j][s], s0);
                acc[j] = s0;
            }
            const float sc = octet_transpose_sum(acc, o) * a.inv_sqrt_d;
            if (keep && row[u] < row1) {
                w.scores[(int64_t)(bh0 + o) * a.row_stride + row[u]] = sc;
                if (count) atomicAdd(&s_hist[o * kHistBins + (ord_key(sc) >> kHistShift)], 1u);
            }
        }
        base += UP * RPP;
        if (base < row1) load(base);
    }
    __syncthreads();
    flush_hist<G>(w, bh0, exmask, s_hist);
}

// scan_segment for the bf16 8-head build on the matrix cores: with 8 query
// vectors per key row the vector-ALU dot products, not HBM, bound the scan, so
// each wave scores 16-key tiles with v_mfma_f32_16x16x32_bf16 (A: 16 key rows x
// 32 dims, B: 32 dims x 16 query columns, of which columns 0 .. a.G-1 are the
// group's heads and the rest repeat head 0; lane l supplies key row and column
// l % 16 for dims 8 (l / 16) .. + 7 of each 32-dim step and receives keys
// 4 (l / 16) .. + 3 of column l % 16).  Two tiles per wave, 256 rows per
// iteration from row0 rounded down to a multiple of 4, so that a lane's four
// scores are one aligned 16-byte store (rows before row0 are scored, neither
// stored nor counted); the next rows' loads are issued before the stores.
template <int D, int G>
__device__ void scan_segment_mfma(const StepArgs &a, const Ws &w, int b, int g, uint32_t exmask,
                                  int64_t row0, int64_t row1, uint32_t *s_hist)
{
    constexpr int KS = D / 32, TW = 2;
    static_assert(G <= 16, "one MFMA column per head");
    constexpr int ROWS = (kScoreThreads / 64) * TW * 16;
    static_assert(D % 32 == 0 && ROWS == 2 * kScanRowsPerIter, "tile geometry");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, col = lane & 15, kq = lane >> 4;
    const int bh0 = b * a.Hq + g * a.G;
    if (a.mode == MODE_SELECT && row0 == 0 && tid == 0) atomicAdd(&w.stats[STAT_SCANS], 1ull);
    const uint16_t *kbase = (const uint16_t *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    bf16x8_t qb[KS];
    {
        const int hj = col < a.G ? col : 0;
        const uint4 *qr = (const uint4 *)((const uint16_t *)a.q + (int64_t)(bh0 + hj) * a.q_head_stride);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qb[ks] = __builtin_bit_cast(bf16x8_t, qr[ks * 4 + kq]);
    }
    // column col's scores are stored when its head is exact, or (in a scan-fed
    // step) reuses in a scanned group; only exact heads are counted
    const bool keep = col < a.G && (((exmask >> col) & 1u) || a.scan_fed);
    const bool count = col < a.G && ((exmask >> col) & 1u);
    float *srow = w.scores + (int64_t)(bh0 + (keep ? col : 0)) * a.row_stride;
    uint32_t *hrow = s_hist + col * kHistBins;
    uint4 kv[TW][KS];
    auto load = [&](int64_t base) {
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            const int64_t r = base + (wave * TW + t) * 16 + col;
            const uint4 *rp = (const uint4 *)(kbase + (r < row1 ? r : row0) * D);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kv[t][ks] = rp[ks * 4 + kq];
        }
    };
    const int64_t start = row0 & ~(int64_t)3;
    load(start);   // the first rows are in flight while the histogram is cleared
    __syncthreads();   // the previous segment's histogram flush is done
    for (int i = tid; i < G * kHistBins; i += kScoreThreads) s_hist[i] = 0u;
    __syncthreads();

    for (int64_t base = start; base < row1; base += ROWS) {
        f32x4_t acc[TW];
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            acc[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8_t, kv[t][ks]), qb[ks], acc[t], 0, 0, 0);
        }
        if (base + ROWS < row1) load(base + ROWS);
        if (keep) {
#pragma unroll
            for (int t = 0; t < TW; ++t) {
                const int64_t r4 = base + (wave * TW + t) * 16 + 4 * kq;   // a multiple of 4
                const float sc[4] = {acc[t][0] * a.inv_sqrt_d, acc[t][1] * a.inv_sqrt_d,
                                     acc[t][2] * a.inv_sqrt_d, acc[t][3] * a.inv_sqrt_d};
                const bool whole = r4 >= row0 && r4 + 3 < row1;
                if (whole) *(float4 *)(srow + r4) = make_float4(sc[0], sc[1], sc[2], sc[3]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (r4 + i >= row0 && r4 + i < row1) {
                        if (!whole) srow[r4 + i] = sc[i];
                        if (count) atomicAdd(&hrow[ord_key(sc[i]) >> kHistShift], 1u);
                    }
                }
            }
        }
    }
    __syncthreads();
    flush_hist<G>(w, bh0, exmask, s_hist);
}

// One contiguous segment [row0, row1) of the rows of KV group (b, g): scores of
// the group's exact heads (bits of exmask), written to `scores` and counted in
// each head's histogram.
template <typename T, int D, int G>
__device__ void scan_segment(const StepArgs &a, const Ws &w, int b, int g, uint32_t exmask,
                             int64_t row0, int64_t row1, uint32_t *s_hist)
{
    if constexpr (sizeof(T) == 2 && G == 8) {
        scan_segment_mfma<D, G>(a, w, b, g, exmask, row0, row1, s_hist);
        return;
    } else if constexpr (G == 8) {
        scan_segment_octet<T, D>(a, w, b, g, exmask, row0, row1, s_hist);
        return;
    }
    using R = RowT<T, D>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int bh0 = b * a.Hq + g * a.G;
    if (a.mode == MODE_SELECT && row0 == 0 && tid == 0) atomicAdd(&w.stats[STAT_SCANS], 1ull);
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    // G >= a.G: the heads past a.G pad the group (they read head 0's query and are
    // never in exmask)
    uint4 qv[G][R::kNV];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const int hj = j < a.G ? j : 0;
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)(bh0 + hj) * a.q_head_stride);
#pragma unroll
        for (int s = 0; s < R::kNV; ++s) qv[j][s] = qr[s * 4 + p];
    }
    // Two key rows per lane per iteration, loaded from clamped (in-bounds) rows.
    uint4 kv[2][R::kNV];
    int64_t row[2];
    auto load = [&](int64_t base) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            row[u] = base + u * kScanRowsPerIter + wave * 16 + rl;
            const uint4 *rp = (const uint4 *)(kbase + (row[u] < row1 ? row[u] : row0) * D);
#pragma unroll
            for (int s = 0; s < R::kNV; ++s) kv[u][s] = rp[s * 4 + p];
        }
    };
    load(row0);   // the first rows are in flight while the histogram is cleared
    __syncthreads();   // the previous segment's histogram flush is done
    for (int i = tid; i < G * kHistBins; i += kScoreThreads) s_hist[i] = 0u;
    __syncthreads();

    for (int64_t base = row0; base < row1;) {
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
            if (row[u] < row1) {
#pragma unroll
                for (int jj = 0; jj < (G + 3) / 4; ++jj) {
                    const int j = jj * 4 + (G == 1 ? 0 : (G == 2 ? (p & 1) : p));
                    const bool mine = G == 1 ? p == 0 : (G == 2 ? p < 2 : true);
                    // stored for exact heads and (scan-fed steps) for the reuse
                    // heads of a scanned group; counted for exact heads only
                    const bool ex = ((exmask >> j) & 1u) != 0u;
                    if (mine && j < a.G && (ex || a.scan_fed)) {
                        const float sc = (jj == 0 ? sc_lo : sc_hi) * a.inv_sqrt_d;
                        w.scores[(int64_t)(bh0 + j) * a.row_stride + row[u]] = sc;
                        if (ex) atomicAdd(&s_hist[j * kHistBins + (ord_key(sc) >> kHistShift)], 1u);
                    }
                }
            }
        }
        base += 2 * kScanRowsPerIter;
        if (base < row1) load(base);
    }
    __syncthreads();
    flush_hist<G>(w, bh0, exmask, s_hist);
}

// Scan block sbk: scores its share of the concatenated rows of the KV groups that
// have an exact head, so that the scan work spreads over all scan blocks however
// many groups need it.  Outside MODE_SELECT every group is exact; in MODE_SELECT
// a head is exact iff rho_max < tau (Eq. 13): its reuse flag, which k_sim sets
// when some block's best similarity reaches tau, is clear.
template <typename T, int D, int G, bool kSelect>
__device__ void scan_block(const StepArgs &a, const Ws &w, const Geometry &geo, int sbk,
                           unsigned char *lds)
{
    constexpr int NT = kScoreThreads;
    const int tid = threadIdx.x;
    const int NG = a.B * a.Hkv;
    const int64_t len = a.len;
    uint32_t *s_hist = (uint32_t *)lds;
    // The groups' rows are laid end to end, each group padded to a multiple of 4
    // rows (len4), so that every segment starts on a multiple of 4; the padding
    // rows are skipped.
    const int64_t len4 = (len + 3) & ~(int64_t)3;
    auto do_span = [&](int n_ex, auto group_of) {
        const int64_t total = (int64_t)n_ex * len4;
        int64_t span = (total + geo.scan_blocks - 1) / geo.scan_blocks;
        span = (span + 2 * kScanRowsPerIter - 1) / (2 * kScanRowsPerIter) * (2 * kScanRowsPerIter);
        int64_t pos = (int64_t)sbk * span;
        const int64_t end = pos + span < total ? pos + span : total;
        while (pos < end) {
            const int e = (int)(pos / len4);
            const int64_t r0 = pos - (int64_t)e * len4;
            const int64_t r1 = (r0 + (end - pos) < len4) ? r0 + (end - pos) : len4;
            if (r0 < len) {
                int gi;
                uint32_t m;
                group_of(e, gi, m);
                scan_segment<T, D, G>(a, w, gi / a.Hkv, gi % a.Hkv, m, r0, r1 < len ? r1 : len, s_hist);
            }
            pos += r1 - r0;
        }
    };
    if constexpr (!kSelect) {
        do_span(NG, [&](int e, int &gi, uint32_t &m) { gi = e; m = (1u << a.G) - 1u; });
    } else {
        __shared__ uint32_t s_reuse[kMaxHeads / 32];
        __shared__ uint32_t s_local[kLocalGroups];   // group * 256 + exact-head mask
        __shared__ uint32_t s_red[NT / 64];
        const int BH = a.B * a.Hq;
        for (int i0 = 0; i0 < BH; i0 += NT) {
            const uint64_t bal = __ballot(i0 + tid < BH && w.reuse[i0 + tid] != 0);
            if ((tid & 63) == 0 && i0 + tid < BH) {
                s_reuse[(i0 + tid) >> 5] = (uint32_t)bal;
                if (i0 + tid + 32 < BH) s_reuse[((i0 + tid) >> 5) + 1] = (uint32_t)(bal >> 32);
            }
        }
        __syncthreads();
        auto mask_of = [&](int gi) {
            uint32_t m = 0u;
            const int head0 = (gi / a.Hkv) * a.Hq + (gi % a.Hkv) * a.G;
#pragma unroll
            for (int j = 0; j < G; ++j) {
                const int head = head0 + j;
                if (j < a.G && !((s_reuse[head >> 5] >> (head & 31)) & 1u)) m |= 1u << j;
            }
            return m;
        };
        if (NG <= 64) {
            // One wave ranks the exact groups with a ballot; no block scans.
            __shared__ int s_nex;
            if (tid < 64) {
                const uint32_t m = tid < NG ? mask_of(tid) : 0u;
                const uint64_t bal = __ballot(m != 0u);
                const int e = __popcll(bal & ((1ull << tid) - 1ull));
                if (tid == 0) s_nex = __popcll(bal);
                if (m != 0u) s_local[e] = (uint32_t)tid * 256u + m;
            }
            __syncthreads();
            const int n_ex64 = s_nex;
            if (n_ex64 == 0) return;
            do_span(n_ex64, [&](int e, int &gi, uint32_t &m) {
                const uint32_t x = s_local[e];
                gi = (int)(x >> 8);
                m = x & 255u;
            });
            return;
        }
        // Pass 1: the number of exact groups, hence this block's rows (with at
        // most NT groups, one pass also ranks them).
        int n_ex = 0;
        uint32_t m0 = 0u;
        int e0 = 0;
        for (int g0 = 0; g0 < NG; g0 += NT) {
            const int gi = g0 + tid;
            const uint32_t m = gi < NG ? mask_of(gi) : 0u;
            uint32_t tot;
            const int e = n_ex + (int)block_excl_scan<NT>(m != 0u ? 1u : 0u, s_red, &tot);
            if (g0 == 0) {
                m0 = m;
                e0 = e;
            }
            n_ex += (int)tot;
        }
        if (n_ex == 0) return;
        const int64_t total = (int64_t)n_ex * len4;   // the same layout as do_span
        int64_t span = (total + geo.scan_blocks - 1) / geo.scan_blocks;
        span = (span + 2 * kScanRowsPerIter - 1) / (2 * kScanRowsPerIter) * (2 * kScanRowsPerIter);
        const int64_t pos0 = (int64_t)sbk * span;
        if (pos0 >= total) return;
        const int64_t end0 = pos0 + span < total ? pos0 + span : total;
        const int e_lo = (int)(pos0 / len4), e_hi = (int)((end0 - 1) / len4);
        // Pass 2: keep the exact groups of ranks e_lo .. e_hi.
        if (NG <= NT && m0 != 0u && e0 >= e_lo && e0 <= e_hi && e0 - e_lo < kLocalGroups)
            s_local[e0 - e_lo] = (uint32_t)tid * 256u + m0;
        int rank0 = 0;
        for (int g0 = 0; NG > NT && g0 < NG; g0 += NT) {
            const int gi = g0 + tid;
            const uint32_t m = gi < NG ? mask_of(gi) : 0u;
            uint32_t tot;
            const int e = rank0 + (int)block_excl_scan<NT>(m != 0u ? 1u : 0u, s_red, &tot);
            if (m != 0u && e >= e_lo && e <= e_hi && e - e_lo < kLocalGroups)
                s_local[e - e_lo] = (uint32_t)gi * 256u + m;
            rank0 += (int)tot;
        }
        __syncthreads();
        // A block's span is at most 512 rows when it is short, or about
        // n_ex / scan_blocks + 1 of len rows, so it touches at most
        // min(256 / len, 8) + 3 groups: s_local never fills.
        do_span(n_ex, [&](int e, int &gi, uint32_t &m) {
            const int at = e - e_lo < kLocalGroups ? e - e_lo : kLocalGroups - 1;
            const uint32_t x = s_local[at];
            gi = (int)(x >> 8);
            m = x & 255u;
        });
    }
}

// Range block s of head bh: path rule, Top-R, the head's candidates inside index
// range s, and their scores.  Entries go to region (bh, s) in index order.
template <typename T, int D>
__device__ void range_block(const StepArgs &a, const Ws &w, int cb, unsigned char *lds)
{
    using R = RowT<T, D>;
    constexpr int NT = kScoreThreads, NW = NT / 64;
    const int kCands = ((a.M + kSimSlots - 1) / kSimSlots) * a.R;   // merge candidates
    __shared__ uint32_t s_red32[NT / 64];
    __shared__ int32_t s_ret[kMaxR];
    __shared__ int32_t s_retcnt[kMaxR];
    __shared__ double s_retrho[kMaxR];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    // the kCandRanges blocks of head bh run on XCD bh % 8 (block j is placed on
    // XCD j % 8), beside the head's similarity blocks and final blocks
    const int xcd = cb & 7, rest = cb >> 3;
    const int s = rest % kCandRanges, bh = (rest / kCandRanges) * 8 + xcd;
    if (bh >= a.B * a.Hq) return;

    const int M = a.M;
    const int n_valid = (int)(a.n_ins < (int64_t)M ? a.n_ins : (int64_t)M);
    const int nsb = (M + kSimSlots - 1) / kSimSlots;
    const int nret_all = a.R < n_valid ? a.R : n_valid;
    double *c_rho = (double *)lds;
    int32_t *c_slot = (int32_t *)(lds + 8 * kCands);
    int32_t *c_cnt = (int32_t *)(lds + 12 * kCands);
    int32_t *c_age = (int32_t *)(lds + 16 * kCands);
    int32_t *c_rank = (int32_t *)(lds + 20 * kCands);
    const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;

    // Retrieved positions no list entry fills stay empty (possible only when the
    // similarities are not ordered, e.g. NaN): they are skipped, never read.
    if (tid < kMaxR) {
        s_ret[tid] = -1;
        s_retcnt[tid] = 0;
        s_retrho[tid] = -INFINITY;
    }
    // Independent loads first: the k_sim blocks' Top-R lists (each one sorted,
    // most similar first, invalid entries last) and q.
    const int per = a.R;                        // list length of a full k_sim block
    const int nc = nsb * per;
    const int age0 = a.insert_slot > 0 ? a.insert_slot - 1 : M - 1;   // slot of the newest entry
    for (int c = tid; c < nc; c += NT) {
        const int sb = c / per, j = c - sb * per;
        const int nloc = n_valid - sb * kSimSlots;
        const bool valid = j < (nloc < kSimSlots ? nloc : kSimSlots);
        const int64_t src = ((int64_t)bh * (kMaxCache / kSimSlots) + sb) * kMaxR + j;
        const int32_t sl = w.topr[src];
        const double rr = w.topr_rho[src];
        const int32_t cn = w.topr_cnt[src];
        const bool use = valid && sl >= 0 && sl < M;   // recent-R lists can be shorter
        c_slot[c] = use ? sl : -1;
        c_rho[c] = use ? rr : -INFINITY;
        c_cnt[c] = use ? cn : 0;
        c_age[c] = use ? slot_age(age0, sl, M) : 0x7FFFFFFF;
        c_rank[c] = 0;
    }
    uint4 qv[R::kNV];
    {
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)bh * a.q_head_stride);
#pragma unroll
        for (int v = 0; v < R::kNV; ++v) qv[v] = qr[v * 4 + p];
    }
    // In a scan-fed step: whether the head's KV group is scanned (some head of the
    // group falls back: its reuse bit is clear), by the rule the scan blocks
    // apply; bit j of s_grp: head j of the group reuses.
    __shared__ uint32_t s_grp;
    if (a.scan_fed && tid == 0) {
        const int head0 = b * a.Hq + g * a.G;
        uint32_t all = 0u;
        for (int j = 0; j < a.G; ++j) all |= (w.reuse[head0 + j] != 0 ? 1u : 0u) << j;
        s_grp = all;
    }
    __syncthreads();

    // Eq. 7 over the k_sim blocks' lists (their union holds the global Top-R):
    // a listed candidate's rank is the number of listed candidates before it --
    // more similar, or equally similar and newer (for recent-R retrieval: newer)
    // -- and ranks 0 .. nret_all-1 are retrieved.  Ages are distinct, so the ranks
    // are; a candidate whose similarity is not ordered (NaN) is never taken.
    // Each wave counts one share of the comparisons; LDS adds the shares.
    {
        const bool recent = a.retrieval == 1;
        const int jper = (nc + NW - 1) / NW;
        const int j0 = wave * jper, j1 = j0 + jper < nc ? j0 + jper : nc;
        for (int c = lane; c < nc; c += 64) {
            const double rc = c_rho[c];
            const int ac = c_age[c];
            int part = 0;
            if (recent) {
                for (int j = j0; j < j1; ++j) part += ((c_slot[j] >= 0) & (c_age[j] < ac)) ? 1 : 0;
            } else {
#pragma unroll 4
                for (int j = j0; j < j1; ++j) {
                    const double rj = c_rho[j];
                    const int aj = c_age[j];
                    const bool ej = (c_slot[j] >= 0) & (rj == rj);
                    part += (ej & ((rj > rc) | ((rj == rc) & (aj < ac)))) ? 1 : 0;
                }
            }
            if (part) atomicAdd(&c_rank[c], part);
        }
    }
    __syncthreads();
    for (int c = tid; c < nc; c += NT) {
        const int rk = c_rank[c];
        const int32_t sl = c_slot[c];
        const double rc = c_rho[c];
        if (sl >= 0 && rc == rc && rk < nret_all) {
            s_ret[rk] = sl;
            s_retcnt[rk] = c_cnt[c];
            s_retrho[rk] = rc;
        }
    }
    __syncthreads();

    // rho_max, the best similarity among the retrieved entries (for Eq. 7 the
    // most similar entry of all), and the path (Eq. 13).
    double mx = -INFINITY;
    for (int i = 0; i < nret_all; ++i) mx = fmax(mx, s_retrho[i]);
    const int8_t path = mx < (double)a.tau ? PATH_FALLBACK : PATH_REUSE;
    const int nret = path == PATH_REUSE ? nret_all : 0;
    // a reuse head of a scanned group: its candidates' scores come from the scan
    const bool from_scan = a.scan_fed && path == PATH_REUSE && s_grp != (1u << a.G) - 1u;
    if (s == 0 && tid == 0) {
        w.path[bh] = from_scan ? PATH_REUSE_SCANNED : path;
        if (a.dbg_path) a.dbg_path[bh] = path;
        if (a.dbg_rho) a.dbg_rho[bh] = mx;
        atomicAdd(&w.stats[path == PATH_REUSE ? STAT_REUSE : STAT_FALLBACK], 1ull);
    }
    if (path != PATH_REUSE) {
        if (s == 0 && a.dbg_ret)
            for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = -1;
        return;
    }
    if (s == 0 && a.dbg_ret)
        for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = i < nret ? s_ret[i] : -1;

    // Eq. 8-9 restricted to this block's index range [lo, hi) of the split the
    // host made for the step (the window's rows in ranges of their own).
    const int64_t len = a.len;
    const int64_t w0 = a.w0;
    const int n_old = kCandRanges - a.n_win;         // ranges covering [0, w0)
    int64_t lo, hi;
    if (s < n_old) {
        lo = (int64_t)s * a.span_old;
        hi = lo + a.span_old < w0 ? lo + a.span_old : w0;
    } else {
        lo = w0 + (int64_t)(s - n_old) * a.span_win;
        hi = lo + a.span_win < len ? lo + a.span_win : len;
    }
    if (lo > hi) lo = hi;
    uint32_t *bitmap = (uint32_t *)lds;                    // reuses the merge space
    int32_t *list = (int32_t *)(lds + kSegWords * 4);
    uint64_t *ents = w.cand_ent + ((int64_t)bh * kCandRanges + s) * a.cand_cap;
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    __syncthreads();   // the merge candidates are dead from here on

    int total = 0;
    for (int64_t seg = lo; seg < hi; seg += (int64_t)kSegWords * 32) {
        const int64_t seg_hi = seg + (int64_t)kSegWords * 32 < hi ? seg + (int64_t)kSegWords * 32 : hi;
        const int nwords = (int)((seg_hi - seg + 31) >> 5);
        // Supports of the retrieved entries: 8 supports' loads in flight before
        // any bitmap update.
        for (int t0 = 0; t0 < a.K; t0 += NT) {
            for (int r0 = 0; r0 < nret; r0 += 8) {
                // Unconditional loads from clamped (in-bounds) addresses, masked
                // afterwards, so that all eight are in flight together.
                int32_t xv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int r = r0 + u < nret ? r0 + u : 0;
                    const int t = t0 + tid < a.K ? t0 + tid : 0;
                    const int32_t sl = s_ret[r];
                    const bool ok = r0 + u < nret && sl >= 0 && t0 + tid < s_retcnt[r];
                    const int32_t x = w.supp[((int64_t)bh * M + (sl >= 0 ? sl : 0)) * a.K + t];
                    xv[u] = ok ? x : -1;
                }
                if (t0 == 0 && r0 == 0) {
                    for (int i = tid; i < nwords; i += NT) bitmap[i] = 0u;
                    __syncthreads();
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int64_t x = xv[u];
                    if (x >= seg && x < seg_hi) atomicOr(&bitmap[(x - seg) >> 5], 1u << ((x - seg) & 31));
                }
            }
        }
        if (nret == 0) {
            for (int i = tid; i < nwords; i += NT) bitmap[i] = 0u;
            __syncthreads();
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
            if (from_scan) {
                // the candidate indices only; k_filter puts in their ranks once the
                // scan has stored the scores
                for (int i = tid; i < nr; i += NT) ents[total + rb + i] = (uint64_t)(uint32_t)list[i];
            }
            // Eq. 10 on this round: 4 lanes per key row, four rows per lane in
            // flight (two for 512-byte rows, whose four would fill the registers),
            // loaded from clamped (in-bounds) list positions.
            constexpr int GU = R::kNV >= 8 ? 2 : 4;
            for (int base = 0; !from_scan && base < nr; base += GU * kScanRowsPerIter) {
                uint4 kv[GU][R::kNV];
                int ci[GU], cidx[GU];
#pragma unroll
                for (int u = 0; u < GU; ++u) {
                    ci[u] = base + u * kScanRowsPerIter + wave * 16 + rl;
                    cidx[u] = list[ci[u] < nr ? ci[u] : nr - 1];
                    const uint4 *rp = (const uint4 *)(kbase + (int64_t)cidx[u] * D);
#pragma unroll
                    for (int v = 0; v < R::kNV; ++v) kv[u][v] = rp[v * 4 + p];
                }
#pragma unroll
                for (int u = 0; u < GU; ++u) {
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

// kSelect: the decode-step variant with range blocks (MODE_SELECT); otherwise
// every head is exact and the grid holds scan blocks only.  Dynamic LDS:
// max(score_scan_lds(G), score_range_lds(merge candidates)) bytes.
template <typename T, int D, int G, bool kSelect>
__global__ __launch_bounds__(kScoreThreads, (kGroupWaves<T, D, G>)) void k_score(StepArgs a, Ws w, Geometry geo)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    // The host orders the two kinds of block (both counts are multiples of 8, so
    // a block's XCD does not depend on the order).
    const int first = kSelect ? (geo.scan_first ? geo.scan_blocks : geo.cand_blocks) : 0;
    const bool is_range = kSelect && (((int)blockIdx.x < first) != (geo.scan_first != 0));
    if (is_range)
        range_block<T, D>(a, w, (int)blockIdx.x - (geo.scan_first ? first : 0), lds);
    else
        scan_block<T, D, G, kSelect>(a, w, geo, (int)blockIdx.x - (kSelect && !geo.scan_first ? first : 0), lds);
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
    // the reuse flags k_sim set for this step were read by k_score; cleared here
    // for the next step
    if (a.mode == MODE_SELECT && blockIdx.x == 0)
        for (int i = tid; i < a.B * a.Hq; i += NT) w.reuse[i] = 0;
    // the filter blocks of (virtual) head vh run on XCD vh % 8 (block j is placed
    // on XCD j % 8), where the head's range blocks wrote its path and candidates
    // and its final blocks read the survivors
    const int x8 = (int)blockIdx.x & 7, rest = (int)blockIdx.x >> 3;
    const int f = rest % geo.filter_blocks_per_head;
    const int vh = (rest / geo.filter_blocks_per_head) * 8 + x8;
    if (vh >= a.B * a.Hq * a.U) return;
    const int64_t len = a.U > 1 ? a.len + vh / (a.B * a.Hq) : a.len;
    if (a.mode == MODE_SELECT) {
        const int8_t path = w.path[vh];
        if (path == PATH_REUSE) return;
        if (path == PATH_REUSE_SCANNED) {
            // Eq. 10 from the scan's scores: the candidate indices of range r
            // (blocks f, f + fpb, ... of the head) become their ranks
            for (int r = f; r < kCandRanges; r += geo.filter_blocks_per_head) {
                uint64_t *ents = w.cand_ent + ((int64_t)vh * kCandRanges + r) * a.cand_cap;
                const int n = (int)w.cand_cnt[(int64_t)vh * kCandRanges + r];
                const float *srow = w.scores + (int64_t)vh * a.row_stride;
                for (int j0 = tid; j0 < n; j0 += 4 * NT) {
                    uint32_t idx[4];
                    float sc[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) idx[u] = (uint32_t)ents[j0 + u * NT < n ? j0 + u * NT : j0];
#pragma unroll
                    for (int u = 0; u < 4; ++u) sc[u] = srow[idx[u]];
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        if (j0 + u * NT < n) ents[j0 + u * NT] = rank_of(sc[u], idx[u]);
                }
            }
            return;
        }
    }

    // This block's scores (or, after k_scan_list, the region's count and its
    // first 2 * NT local survivors) and the head's histogram in one round trip.
    const int64_t i0 = (int64_t)f * kFilterRows + (int64_t)tid * EPT;
    uint64_t *reg = w.surv + (int64_t)vh * a.row_stride + (int64_t)f * kFilterRows;
    float4 v0, v1;
    uint4 lv, lv2 = {};
    uint32_t nloc = 0u;
    // after k_scan_list, a whole region holds its local survivors; the rows past
    // the last whole region are in the score row
    const bool listed = geo.list_mode && f < (int)(len / kFilterRows);
    if (listed) {
        nloc = w.surv_cnt[(int64_t)vh * a.n_regions + f];
        if (a.K > 512) {
            lv = ((const uint4 *)reg)[2 * tid];
            lv2 = ((const uint4 *)reg)[2 * tid + 1];
        } else {
            lv = ((const uint4 *)reg)[tid];
        }
    } else {
        const float4 *src = (const float4 *)(w.scores + (int64_t)vh * a.row_stride + i0);
        v0 = src[0];
        v1 = src[1];
    }
    const uint32_t *hist = w.hist + (int64_t)vh * kHistBins;
    uint32_t c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = hist[kHistBins - 1 - 4 * tid - j];

    // The bin b* that holds the kn-th largest score: the largest b with
    // count(bins >= b) >= kn.  Thread t holds bins 2047-4t .. 2044-4t.
    {
        const uint32_t kn = (uint32_t)(a.K < len ? a.K : len);
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
    if (listed) {
        // The region's local survivors at or above b*, compacted in place in
        // index order: thread t holds entries m t .. m t + m-1, with m = 2 (4 for
        // K > 512) from the first round trip, or m = 8 when the region kept more,
        // all read before the scan's barriers.
        uint64_t e[EPT] = {};
        int m = a.K > 512 ? 4 : 2;
        if (nloc <= (uint32_t)(m * NT)) {
            e[0] = ((uint64_t)lv.y << 32) | lv.x;
            e[1] = ((uint64_t)lv.w << 32) | lv.z;
            e[2] = ((uint64_t)lv2.y << 32) | lv2.x;
            e[3] = ((uint64_t)lv2.w << 32) | lv2.z;
        } else {
            m = EPT;
#pragma unroll
            for (int u = 0; u < EPT / 2; ++u) {
                const uint4 x = ((const uint4 *)reg)[EPT / 2 * tid + u];
                e[2 * u] = ((uint64_t)x.y << 32) | x.x;
                e[2 * u + 1] = ((uint64_t)x.w << 32) | x.z;
            }
        }
        uint32_t keep = 0, n = 0;
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const bool k = u < m && (uint32_t)(m * tid + u) < nloc && rank_key(e[u]) >= kmin;
            keep |= (uint32_t)k << u;
            n += k ? 1u : 0u;
        }
        uint32_t total;
        uint32_t pos = block_excl_scan<NT>(n, s_red, &total);
#pragma unroll
        for (int u = 0; u < EPT; ++u)
            if ((keep >> u) & 1u) reg[pos++] = e[u];
        if (tid == 0) w.surv_cnt[(int64_t)vh * a.n_regions + f] = total;
        return;
    }
    const float sv[EPT] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint32_t keep = 0, n = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const bool k = i0 + e < len && ord_key(sv[e]) >= kmin;
        keep |= (uint32_t)k << e;
        n += k ? 1u : 0u;
    }
    uint32_t total;
    uint32_t pos = block_excl_scan<NT>(n, s_red, &total);
    uint64_t *dst = w.surv + (int64_t)vh * a.row_stride + (int64_t)f * kFilterRows;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
        if ((keep >> e) & 1u) dst[pos++] = rank_of(sv[e], (uint32_t)(i0 + e));
    if (tid == 0) w.surv_cnt[(int64_t)vh * a.n_regions + f] = total;
}

// ---------------------------------------------------------------------------
// k_final
// ---------------------------------------------------------------------------

constexpr int kTieMax = 64;        // bin sizes resolved by one wave
constexpr int kSpecLoads = 4;      // speculative entry loads per thread

template <int D, int DS, int NT>
struct FinalSmem {
    uint64_t ent[kEntCache];        // the head's entries in index order, when they fit
    uint64_t sel[kMaxK];            // selected (index << 32 | score key), index order
    uint32_t pref[kMaxRegions + 1]; // region prefix counts
    uint32_t hist[kHistBins];
    float part[NT / 64][DS];
    float lpart[NT / 64];
    float qbar[D];
    double red64[NT / 64];
    uint32_t redu[NT / 64];
    uint32_t wcnt[NT / 64];         // per-wave counts of the ordered compaction
    uint64_t tie[kTieMax];          // entries of the bin that holds the K-th largest
    unsigned long long rmax, rmin;
    uint64_t thr;
    uint32_t found_digit, found_above, found_cnt, n_tie;
};

// Entries of one head, spread over regions of a fixed stride, read in order.
struct Regions {
    const uint64_t *base;
    int64_t stride;
    int n;
    const uint64_t *staged;   // LDS copy or nullptr
    const uint32_t *pref;
    int nreg;
    int top;                  // largest power of two below nreg (0 if nreg == 1)
    __device__ uint64_t get(int j) const
    {
        if (staged) return staged[j];
        int lo = 0;           // last region r with pref[r] <= j (empty regions skipped)
        for (int step = top; step > 0; step >>= 1) {
            const int c = lo + step;
            if (c < nreg && (int)pref[c] <= j) lo = c;
        }
        return base[(int64_t)lo * stride + (j - (int)pref[lo])];
    }
};

// Descending scan of sm.hist (nb <= kHistBins bins): the bin where the count
// from the top reaches k (found_digit), the count above it and its own count.
// Thread t covers bins nb-1-BPT*t .. nb-BPT-BPT*t.
template <class SM, int NT>
__device__ void find_bin(SM &sm, uint32_t nb, uint32_t k)
{
    constexpr int BPT = (kHistBins + NT - 1) / NT;
    const int tid = threadIdx.x;
    uint32_t c[BPT], mine = 0;
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
        const int dgt = (int)nb - 1 - BPT * tid - j;
        c[j] = dgt >= 0 ? sm.hist[dgt] : 0u;
        mine += c[j];
    }
    uint32_t all;
    uint32_t above = block_excl_scan<NT>(mine, sm.redu, &all);
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
        if (above < k && above + c[j] >= k) {
            sm.found_digit = nb - 1u - (uint32_t)(BPT * tid + j);
            sm.found_above = above;
            sm.found_cnt = c[j];
        }
        above += c[j];
    }
    __syncthreads();
}

// Radix select over distinct 64-bit ranks with 11-bit digits, most significant
// first, starting at the highest bit in which the ranks differ (rmax ^ rmin).
// On return the top min(K, n) entries are exactly those with
// (rank & mask) >= prefix (mask == 0 selects everything).
template <class SM, int NT>
__device__ void radix_threshold(const Regions &rg, int K, SM &sm, uint64_t &prefix,
                                uint64_t &mask)
{
    const int tid = threadIdx.x;
    prefix = 0;
    mask = 0;
    if (rg.n <= K) return;
    const uint64_t diff = (uint64_t)sm.rmax ^ (uint64_t)sm.rmin;   // nonzero: ranks are distinct
    const int hb = 63 - __clzll((long long)diff);
    if (hb < 63) {
        mask = ~0ull << (hb + 1);
        prefix = (uint64_t)sm.rmax & mask;
    }
    uint32_t k_rem = (uint32_t)K;
    for (int top = hb; top >= 0; top -= 11) {
        const int width = top + 1 < 11 ? top + 1 : 11;
        const int sh = top + 1 - width;
        const uint32_t nb = 1u << width;
        for (uint32_t i = tid; i < nb; i += NT) sm.hist[i] = 0u;
        __syncthreads();
        for (int j = tid; j < rg.n; j += NT) {
            const uint64_t e = rg.get(j);
            if ((e & mask) == prefix) atomicAdd(&sm.hist[(uint32_t)(e >> sh) & (nb - 1u)], 1u);
        }
        __syncthreads();
        find_bin<SM, NT>(sm, nb, k_rem);
        k_rem -= sm.found_above;
        prefix |= (uint64_t)sm.found_digit << sh;
        mask |= (uint64_t)(nb - 1u) << sh;
        const bool done = sm.found_cnt == k_rem || sh == 0;
        __syncthreads();
        if (done) break;
    }
}

// Threshold rank of the Top-K over the n staged entries (n > K): the K-th largest
// rank, so that the Top-K are exactly the entries e >= thr.  One histogram pass
// over kHistBins bins that are linear in the score between the smallest and the
// largest score (monotone in the score, so every entry of a higher bin outranks
// every entry of a lower one); the K-th largest then lies in one bin, whose
// entries one wave ranks exactly when there are at most kTieMax of them.  Returns
// false when that bin is larger (heavy ties), leaving the radix select to decide.
template <class SM, int NT>
__device__ bool value_threshold(const uint64_t *ent, int n, int K, SM &sm,
                                uint64_t &thr)
{
    const int tid = threadIdx.x, lane = tid & 63;
    const float smax = key_score(rank_key((uint64_t)sm.rmax));
    const float smin = key_score(rank_key((uint64_t)sm.rmin));
    const float range = smax - smin;
    if (!(range > 0.0f) || !(range < 3.0e38f)) return false;   // block-uniform
    const float scale = (float)(kHistBins - 1) / range;
    auto bin_of = [&](uint64_t e) {
        const float sc = key_score(rank_key(e));
        return min((int)((sc - smin) * scale), kHistBins - 1);
    };
    // four entries per thread in flight (LDS reads issued before their use)
    for (int j0 = tid; j0 < n; j0 += 4 * NT) {
        uint64_t e[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) e[u] = ent[j0 + u * NT < n ? j0 + u * NT : j0];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (j0 + u * NT < n) atomicAdd(&sm.hist[bin_of(e[u])], 1u);
    }
    __syncthreads();
    find_bin<SM, NT>(sm, kHistBins, (uint32_t)K);
    const uint32_t bstar = sm.found_digit, cnt = sm.found_cnt;
    const uint32_t k_rem = (uint32_t)K - sm.found_above;
    if (cnt > (uint32_t)kTieMax) return false;
    for (int j0 = tid; j0 < n; j0 += 4 * NT) {
        uint64_t e[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) e[u] = ent[j0 + u * NT < n ? j0 + u * NT : j0];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (j0 + u * NT < n && (uint32_t)bin_of(e[u]) == bstar)
                sm.tie[atomicAdd(&sm.n_tie, 1u)] = e[u];
    }
    __syncthreads();
    if (tid < 64) {
        const uint64_t e = lane < (int)cnt ? sm.tie[lane] : 0ull;
        uint32_t above = 0;
        for (int i = 0; i < (int)cnt; ++i) above += sm.tie[i] > e ? 1u : 0u;
        if (lane < (int)cnt && above == k_rem - 1u) sm.thr = e;
    }
    __syncthreads();
    thr = sm.thr;
    return true;
}

// ---------------------------------------------------------------------------
// k_final fast path (decode steps and Exact Top-K): the head's entries stay in
// registers, up to kFastEPT consecutive ones per thread (thread order is index
// order), loaded with the region counts in one round trip when the speculation
// holds, else in a second one; every wave derives the region offsets and the
// threshold bin itself; the selected entries go to an index-ordered list in LDS,
// from which dense row loads feed Softmax-V.  Heads that do not fit (more than
// kFastRegions regions, more entries than the threads can hold, a degenerate
// score range, or more than kTieMax entries in the threshold bin after two levels
// of bins) take the general path below, which reloads everything.
// ---------------------------------------------------------------------------


constexpr int kFastBins = 512;                         // value-linear score bins
constexpr int kFastRegions = 64;                       // regions one wave ranks


struct FastSmem {
    uint32_t hist[kFastBins];
    uint64_t tie[kTieMax + 64];     // the final bin's entries, then one spare slot a lane
    uint32_t wmax[kFinalThreads / 64], wmin[kFinalThreads / 64];
    uint32_t wsel[kFinalThreads / 64];
    uint32_t n_tie;
};

// The bin b* that holds the k-th largest of the entries counted in hist (nb bins,
// descending from bin nb - 1), the count above it and its own count, found by one
// wave (every wave gets the same result): lane l sums bins nb-1-BPL*l ..
// nb-BPL-BPL*l, a wave prefix sum finds the lane, that lane walks its bins.
template <int NB>
__device__ __forceinline__ void wave_find_bin(const uint32_t *hist, uint32_t k, uint32_t &bstar,
                                              uint32_t &above, uint32_t &cnt)
{
    constexpr int BPL = NB / 64;
    static_assert(BPL % 4 == 0, "whole 16-byte reads");
    const int lane = threadIdx.x & 63;
    uint32_t c[BPL], mine = 0u;
    const uint4 *hv = (const uint4 *)&hist[NB - BPL * (lane + 1)];
#pragma unroll
    for (int i = 0; i < BPL / 4; ++i) {
        const uint4 x = hv[i];
        c[BPL - 1 - 4 * i] = x.x;
        c[BPL - 2 - 4 * i] = x.y;
        c[BPL - 3 - 4 * i] = x.z;
        c[BPL - 4 - 4 * i] = x.w;
    }
#pragma unroll
    for (int i = 0; i < BPL; ++i) mine += c[i];
    const uint32_t inc = wave_incl_scan(mine);
    const uint64_t hit = __ballot(inc - mine < k && inc >= k);
    const int src = __builtin_ctzll(hit);   // k <= total: exactly one lane
    uint32_t bs = 0u, ab = 0u, cb = 0u, run = inc - mine;
#pragma unroll
    for (int i = 0; i < BPL; ++i) {
        if (run < k && run + c[i] >= k) {
            bs = (uint32_t)(NB - 1 - BPL * lane - i);
            ab = run;
            cb = c[i];
        }
        run += c[i];
    }
    bstar = (uint32_t)__builtin_amdgcn_readlane((int)bs, src);
    above = (uint32_t)__builtin_amdgcn_readlane((int)ab, src);
    cnt = (uint32_t)__builtin_amdgcn_readlane((int)cb, src);
}

// Block (bh, slice) of k_final on the fast path, one of NS slice blocks of the
// head, holding up to EPT entries per thread.  Returns false, with every thread
// agreeing and nothing written yet, when the head must take the general path.
template <typename T, int D, int NS, int EPT>
__device__ bool final_fast(const StepArgs &a, const Ws &w, int bh, int slice, FastSmem &fs,
                           uint64_t *stage, uint64_t *list, float (*part)[D / NS + 1])
{
    constexpr int NT = kFinalThreads, NW = NT / 64;
    constexpr int kFastSlots = NT * EPT;                  // entries one block holds
    constexpr int DS = D / NS;                            // elements of this block's slice
    constexpr int EPV = 16 / (int)sizeof(T);
    constexpr int LPR = DS * (int)sizeof(T) / 16;         // lanes per slice row
    constexpr int RPW = 64 / LPR;                         // rows per wave instruction
    static_assert(LPR >= 1 && LPR <= 16 && DS * (int)sizeof(T) == LPR * 16, "slice geometry");
    static_assert(EPT <= 32 && EPT % 2 == 0, "entry masks");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool sel_mode = a.mode == MODE_SELECT;
    const int64_t len = a.len;
    const int nreg_x = (int)((len + kFilterRows - 1) / kFilterRows);   // exact layout
    // which of the head's closing writes this block owns (shared out over its slices)
    const bool own_sel = slice == 0, own_supp = (1 % NS) == slice;
    const bool own_qbar = (2 % NS) == slice, own_misc = (3 % NS) == slice;
    // the normalised query k_sim stored, for the cache entry: loaded with the first
    // round trip so that the closing writes wait for no load
    static_assert(D <= NT, "one element per thread");
    const float qcur = a.do_insert && own_qbar && sel_mode && tid < D ? w.qbar_cur[(int64_t)bh * D + tid] : 0.0f;

    for (int i = tid; i < kFastBins; i += NT) fs.hist[i] = 0u;
    if (tid == 0) fs.n_tie = 0u;

    // Entries in registers, thread order = index order: thread t holds entries
    // j0 .. j0+EPT-1 of region r_me (regions in index order, entries ascending),
    // each region taking ceil(count / EPT) consecutive threads, so the live
    // entries sit in the first threads and the other waves skip the per-entry
    // work.  First round trip: the path, the counts of both layouts and,
    // speculatively, EPT entries per thread of the expected layout (the candidate
    // ranges for a decode step that selects, the survivor regions otherwise),
    // each region taking an equal share of the slots.  When the speculation holds,
    // its entries are repacked through LDS; when the head's layout is the other
    // one, or a region holds more entries than its share, a second round trip
    // loads exactly the live entries.
    const int8_t path = sel_mode ? w.path[bh] : (int8_t)PATH_FALLBACK;
    uint64_t e[EPT];
#pragma unroll
    for (int u = 0; u < EPT; ++u) e[u] = 0ull;
    const uint32_t cnt_r = lane < kCandRanges ? w.cand_cnt[(int64_t)bh * kCandRanges + lane] : 0u;
    const uint32_t cnt_x = lane < (nreg_x < kFastRegions ? nreg_x : kFastRegions)
                               ? w.surv_cnt[(int64_t)bh * a.n_regions + lane] : 0u;
    bool reuse = sel_mode;
    const uint64_t *base = reuse ? w.cand_ent + (int64_t)bh * kCandRanges * a.cand_cap
                                 : w.surv + (int64_t)bh * a.row_stride;
    int64_t stride = reuse ? a.cand_cap : kFilterRows;
    int nreg = reuse ? kCandRanges : nreg_x;
    if (nreg > kFastRegions) return false;
    bool staged = false;
    {
        const int spec = (int)((kFastSlots / nreg < stride ? kFastSlots / nreg : stride) &
                               ~(int64_t)(EPT - 1));
        const int slot = tid * EPT;
        const int rs = spec > 0 ? slot / spec : nreg;
        const int js = slot - (rs < nreg ? rs : 0) * spec;
        if (rs < nreg) {
            const uint64_t *src = base + (int64_t)rs * stride + js;
            if ((stride & 1) == 0) {
                // 16-byte aligned: regions start on even entries, js is a multiple of EPT
#pragma unroll
                for (int u = 0; u < EPT / 2; ++u) {
                    const uint4 x = ((const uint4 *)src)[u];
                    e[2 * u] = ((uint64_t)x.y << 32) | x.x;
                    e[2 * u + 1] = ((uint64_t)x.w << 32) | x.z;
                }
            } else {
#pragma unroll
                for (int u = 0; u < EPT; ++u) e[u] = src[u];
            }
        }
        const uint32_t rc = reuse ? cnt_r : cnt_x;
        const bool fits = spec > 0 && __ballot(lane < nreg && rc > (uint32_t)spec) == 0ull;
        if (sel_mode && path != PATH_REUSE && path != PATH_REUSE_SCANNED) {
            reuse = false;
            base = w.surv + (int64_t)bh * a.row_stride;
            stride = kFilterRows;
            nreg = nreg_x;
            if (nreg > kFastRegions) return false;
        } else if (fits) {
            // stage the speculative entries in index order
            const uint32_t inc = wave_incl_scan(rc);
            const uint32_t rpref = (uint32_t)__shfl((int)(inc - rc), rs < nreg ? rs : 0);
            const uint32_t rcnt_s = (uint32_t)__shfl((int)rc, rs < nreg ? rs : 0);
#pragma unroll
            for (int u = 0; u < EPT; ++u)
                if (rs < nreg && (uint32_t)(js + u) < rcnt_s) stage[rpref + js + u] = e[u];
            staged = true;
            __syncthreads();                                          // barrier 0
        }
    }
    const uint32_t rcnt = reuse ? cnt_r : cnt_x;      // lane r: count of region r
    const uint32_t incl = wave_incl_scan(rcnt);
    const uint32_t n = (uint32_t)__builtin_amdgcn_readlane((int)incl, nreg - 1);
    if (n == 0u) return false;
    // p0: the index-order position of this thread's first entry; nlive: how many
    // of its entries are live (they are the first ones)
    uint32_t p0 = 0u, nlive = 0u;
    if (staged) {
        // the staged list is dense: thread t takes positions EPT*t .. EPT*t+EPT-1
        p0 = (uint32_t)(tid * EPT);
        nlive = p0 < n ? (n - p0 < (uint32_t)EPT ? n - p0 : (uint32_t)EPT) : 0u;
#pragma unroll
        for (int u = 0; u < EPT; ++u)
            if ((uint32_t)u < nlive) e[u] = stage[p0 + u];
    } else {
        // region r gets ceil(count / EPT) threads, from thread start tincl[r] - need[r]
        const uint32_t need = lane < nreg ? (rcnt + EPT - 1) / EPT : 0u;
        const uint32_t tincl = wave_incl_scan(need);
        const uint32_t tall = (uint32_t)__builtin_amdgcn_readlane((int)tincl, 63);
        if (tall > (uint32_t)NT) return false;
        int lo = 0;   // the last region whose thread start is <= tid
#pragma unroll
        for (int step = 32; step > 0; step >>= 1) {
            const int c = lo + step;
            const uint32_t st = (uint32_t)__shfl((int)(tincl - need), c < 64 ? c : 63);
            if (c < nreg && st <= (uint32_t)tid) lo = c;
        }
        // the shuffles read lane lo, so every lane takes part (a lane outside the
        // branch below may be the one read)
        const uint32_t st0 = (uint32_t)__shfl((int)(tincl - need), lo);
        const uint32_t rc = (uint32_t)__shfl((int)rcnt, lo);
        const uint32_t rpos = (uint32_t)__shfl((int)(incl - rcnt), lo);
        const uint32_t j0 = ((uint32_t)tid - st0) * EPT;
        if ((uint32_t)tid < tall && j0 < rc) {
            p0 = rpos + j0;
            nlive = rc - j0 < (uint32_t)EPT ? rc - j0 : (uint32_t)EPT;
            const uint64_t *src = base + (int64_t)lo * stride + j0;
            if ((stride & 1) == 0) {
#pragma unroll
                for (int u = 0; u < EPT / 2; ++u) {
                    if ((uint32_t)(2 * u) < nlive) {
                        const uint4 x = ((const uint4 *)src)[u];
                        e[2 * u] = ((uint64_t)x.y << 32) | x.x;
                        e[2 * u + 1] = ((uint64_t)x.w << 32) | x.z;
                    }
                }
            } else {
#pragma unroll
                for (int u = 0; u < EPT; ++u)
                    if ((uint32_t)u < nlive) e[u] = src[u];
            }
        }
    }
    uint32_t valid = (1u << nlive) - 1u;   // bit u: entry u of this thread is a live entry
    // waves holding no entry skip the per-entry work (a wave-uniform branch)
    const bool wlive = __ballot(valid != 0u) != 0ull;

    // the largest and smallest score key
    uint32_t kmax = 0u, kmin = 0xFFFFFFFFu;
    if (wlive) {
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            if ((valid >> u) & 1u) {
                kmax = max(kmax, rank_key(e[u]));
                kmin = min(kmin, rank_key(e[u]));
            }
        }
    }
    kmax = wave_max_u32(kmax);
    kmin = ~wave_max_u32(~kmin);
    if (lane == 0) {
        fs.wmax[wave] = kmax;
        fs.wmin[wave] = kmin;
    }
    __syncthreads();                                                  // barrier 1
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        kmax = max(kmax, fs.wmax[i]);
        kmin = min(kmin, fs.wmin[i]);
    }
    const float smax = key_score(kmax), smin = key_score(kmin);
    const int K = a.K;
    const uint32_t kn = n < (uint32_t)K ? n : (uint32_t)K;

    // Top-K (Eq. 1 / Eq. 11): the entries e >= thr.  Bins linear in the score
    // between the smallest and the largest (monotone in the rank) locate the K-th
    // largest in one bin; when that bin holds more than kTieMax entries, a second
    // level of bins linear over the bin's own score range narrows it; the final
    // bin's entries are ranked exactly by every wave.
    uint64_t thr = 0ull;
    if (n > (uint32_t)K) {
        const float range = smax - smin;
        if (!(range > 0.0f) || !(range < 3.0e38f)) return false;
        float lo = smin, scale = (float)(kFastBins - 1) / range;
        uint32_t cand = valid;     // entries still in the running
        uint32_t k_rem = (uint32_t)K, cnt_b = 0u;
        uint32_t above_mask = 0u;  // entries already known to be in the Top-K
        for (int level = 0; level < 2; ++level) {
            uint32_t bin[EPT];
#pragma unroll
            for (int u = 0; u < EPT; ++u) bin[u] = 0u;
            if (wlive) {
#pragma unroll
                for (int u = 0; u < EPT; ++u) {
                    bin[u] = (uint32_t)min(max((int)((key_score(rank_key(e[u])) - lo) * scale), 0),
                                           kFastBins - 1);
                    if ((cand >> u) & 1u) atomicAdd(&fs.hist[bin[u]], 1u);
                }
            }
            __syncthreads();                                          // barrier 2
            uint32_t bstar, above;
            wave_find_bin<kFastBins>(fs.hist, k_rem, bstar, above, cnt_b);
            uint32_t in_b = 0u;
            if (wlive) {
                // branch-free: masks by selects
#pragma unroll
                for (int u = 0; u < EPT; ++u) {
                    const uint32_t bit = cand & (1u << u);
                    above_mask |= bin[u] > bstar ? bit : 0u;
                    in_b |= bin[u] == bstar ? bit : 0u;
                }
            }
            cand = in_b;
            k_rem -= above;
            if (cnt_b <= (uint32_t)kTieMax || level == 1) break;
            // second level over the bin's score range (the bin's entries only)
            __syncthreads();   // every wave has read the first-level histogram
            for (int i = tid; i < kFastBins; i += NT) fs.hist[i] = 0u;
            const float w0 = lo + (float)bstar / scale;
            lo = w0;
            scale = scale * (float)(kFastBins - 1);
            __syncthreads();
        }
        if (cnt_b > (uint32_t)kTieMax) return false;
        // the final bin's entries to LDS: a wave's slots from a prefix sum of its
        // lanes' counts and one reservation; entries outside the bin go to the
        // lane's spare slot, so that the writes need no branches
        if (wlive) {
            const uint32_t mine = (uint32_t)__popc(cand);
            const uint32_t inc = wave_incl_scan(mine);
            const uint32_t wtot = (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
            uint32_t wbase = 0u;
            if (wtot != 0u) {
                if (lane == 63) wbase = atomicAdd(&fs.n_tie, wtot);
                wbase = (uint32_t)__builtin_amdgcn_readlane((int)wbase, 63);
            }
            uint32_t at = wbase + inc - mine;
#pragma unroll
            for (int u = 0; u < EPT; ++u) {
                const bool in = ((cand >> u) & 1u) != 0u;
                fs.tie[in ? at : (uint32_t)(kTieMax + lane)] = e[u];
                at += in ? 1u : 0u;
            }
        }
        __syncthreads();                                              // barrier 3
        // every wave that holds entries ranks the bin's entries (lane i holds entry
        // i, the others are read as scalars): the k_rem-th largest is the threshold;
        // selected are every entry above the final bin and those of it at or above
        // the threshold
        if (wlive) {
            const uint64_t x = lane < (int)cnt_b ? fs.tie[lane] : 0ull;
            const uint32_t xlo = (uint32_t)x, xhi = (uint32_t)(x >> 32);
            uint32_t higher = 0u;
            for (int i = 0; i < (int)cnt_b; ++i) {
                const uint32_t ylo = (uint32_t)__builtin_amdgcn_readlane((int)xlo, i);
                const uint32_t yhi = (uint32_t)__builtin_amdgcn_readlane((int)xhi, i);
                higher += (yhi > xhi || (yhi == xhi && ylo > xlo)) ? 1u : 0u;
            }
            const uint64_t at = __ballot(lane < (int)cnt_b && higher == k_rem - 1u);
            const int tl = __builtin_ctzll(at);
            thr = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)xhi, tl) << 32) |
                  (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)xlo, tl);
#pragma unroll
            for (int u = 0; u < EPT; ++u) above_mask |= (cand & (1u << u)) && e[u] >= thr ? 1u << u : 0u;
        }
        valid = above_mask;
    }
    // No early exit from here on: the counters of a reuse head, or the reset of an
    // exact head's histogram (read by k_filter, the previous launch) for the next
    // launch, go out now so that their latency overlaps the rest.
    if (own_misc) {
        if (reuse) {
            if (tid == 0) {
                atomicAdd(&w.stats[STAT_CAND_SUM], (unsigned long long)n);
                atomicMax(&w.stats[STAT_CAND_MAX], (unsigned long long)n);
            }
        } else {
            for (int i = tid; i < kHistBins; i += NT) w.hist[(int64_t)bh * kHistBins + i] = 0u;
        }
    }
    const uint32_t selm = valid;
    const uint32_t nsel = (uint32_t)__popc(selm);

    // The selected entries in index order (the threads hold consecutive entries):
    // each thread's position from a block scan of the per-thread counts, then the
    // list in LDS, as (index << 32 | score key).
    const uint32_t winc = wave_incl_scan(nsel);
    if (lane == 63) fs.wsel[wave] = winc;
    __syncthreads();                                                  // barrier 4
    uint32_t pos = winc - nsel;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) pos += ww < wave ? fs.wsel[ww] : 0u;
    if (wlive) {
#pragma unroll
        for (int u = 0; u < EPT; ++u)
            if ((selm >> u) & 1u) list[pos++] = ((uint64_t)rank_index(e[u]) << 32) | rank_key(e[u]);
    }
    __syncthreads();                                                  // barrier 5

    // Eq. 12 on this block's slice: weights exp(s - max), the largest selected score
    // being the largest of all.  LPR lanes per value row, RPW rows per wave
    // instruction, four rows per lane in flight.
    {
        const int b = bh / a.Hq, g = (bh % a.Hq) / a.G;
        const T *vbase = (const T *)a.v + ((int64_t)b * a.Hkv + g) * a.max_len * D + slice * DS;
        const int sub = lane / LPR, vl = lane % LPR;
        float acc[EPV], lsum = 0.0f;
#pragma unroll
        for (int i = 0; i < EPV; ++i) acc[i] = 0.0f;
        for (int t0 = wave * RPW + sub; t0 < (int)kn; t0 += 4 * NW * RPW) {
            uint4 raw[4];
            float wt[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int t = t0 + q * NW * RPW;
                const uint64_t se = list[t < (int)kn ? t : 0];
                raw[q] = ((const uint4 *)(vbase + (int64_t)(uint32_t)(se >> 32) * D))[vl];
                wt[q] = t < (int)kn ? expf(key_score((uint32_t)se) - smax) : 0.0f;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                Dot<T>::axpy(raw[q], wt[q], acc);
                lsum += vl == 0 ? wt[q] : 0.0f;
            }
        }
        // sum over the lanes of each row that hold the same vl (row rotations), then
        // over the rows of the block in LDS
#pragma unroll
        for (int o = LPR; o < 16; o <<= 1) {
#pragma unroll
            for (int i = 0; i < EPV; ++i) acc[i] += row_ror_f32(acc[i], o);
            lsum += row_ror_f32(lsum, o);
        }
        const int row = wave * 4 + (lane >> 4);
        if ((lane & 15) < LPR) {
#pragma unroll
            for (int i = 0; i < EPV; ++i) part[row][vl * EPV + i] = acc[i];
            if (vl == 0) part[row][DS] = lsum;
        }
    }
    __syncthreads();                                                  // barrier 6
    if (tid < DS) {
        float o = 0.0f, l = 0.0f;
#pragma unroll
        for (int r = 0; r < 4 * NW; ++r) {
            o += part[r][tid];
            l += part[r][DS];
        }
        a.out[(int64_t)bh * D + slice * DS + tid] = o / l;
    }

    const int64_t ent = (int64_t)bh * a.M + a.insert_slot;   // the cache entry written
    auto put = [&](int32_t *dst) {
        for (int t = tid; t < K; t += NT) dst[t] = t < (int)kn ? (int32_t)(list[t] >> 32) : -1;
    };
    if (own_sel) {
        if (a.sel != nullptr) put(a.sel + (int64_t)bh * K);
        if (a.dbg_ncand && tid == 0) a.dbg_ncand[bh] = reuse ? (int32_t)n : 0;
        if (a.dbg_cand) {
            int32_t *dc = a.dbg_cand + (int64_t)bh * a.cand_cap;
            if (reuse) {
#pragma unroll
                for (int u = 0; u < EPT; ++u)
                    if ((uint32_t)u < nlive) dc[p0 + u] = (int32_t)rank_index(e[u]);
            }
            for (int j = (reuse ? (int)n : 0) + tid; j < a.cand_cap; j += NT) dc[j] = -1;
        }
    }
    if (a.do_insert) {
        // Sec. 3.4: insert (q_bar, support) after either path
        if (own_supp) {
            put(w.supp + ent * K);
            if (tid == 0) w.cnt[ent] = (int32_t)kn;
        }
        if (own_qbar) {
            if (sel_mode) {
                if (tid < D) w.qbar[ent * D + tid] = qcur;
            } else {
                __shared__ float s_qbar[D];
                __shared__ double s_red[NT / 64];
                block_qbar<T, D, NT>((const T *)a.q + (int64_t)bh * a.q_head_stride, s_qbar, s_red);
                for (int t = tid; t < D; t += NT) w.qbar[ent * D + t] = s_qbar[t];
            }
        }
    }
    return true;
}

// kMulti: built for launches of several query positions (a.U > 1, the batched
// prefill); the decode-step build keeps u = 0 out of its code.
template <typename T, int D, bool kMulti, int NSL, int EPT>
__global__ __launch_bounds__(kFinalThreads) void k_final(StepArgs a, Ws w)
{
    constexpr int NT = kFinalThreads;
    constexpr int NW = NT / 64;
    // the multi-position (prefill) build writes no output: one block per head
    constexpr int NS = kMulti ? 1 : NSL;
    constexpr int DS = D / NSL;                          // elements per slice
    constexpr int SB = DS * (int)sizeof(T);              // bytes per slice row
    constexpr int LPR = SB / 16;                         // lanes per slice row
    constexpr int RPW = 64 / LPR;                        // rows per wave instruction
    constexpr int EPV = 16 / (int)sizeof(T);
    constexpr int kRegPerThread = kMaxRegions / NT;
    static_assert(SB % 16 == 0 && LPR >= 1 && LPR <= 64, "slice geometry");
    static_assert(kMaxRegions % NT == 0 && kCandRanges <= NT, "region ownership");
    __shared__ FinalSmem<D, DS, NT> sm;
    __shared__ FastSmem fs;
    __shared__ float s_part[4 * (NT / 64)][DS + 1];
    static_assert(NT * EPT <= kEntCache, "the fast path stages its entries in sm.ent");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int vh, slice;
    if constexpr (kMulti) {
        vh = blockIdx.x;
        slice = 0;
    } else {
        // the NS blocks of head vh run on XCD vh % 8 (block j is placed on XCD
        // j % 8), beside the range blocks that wrote the head's candidates
        const int x = (int)blockIdx.x & 7, rest = (int)blockIdx.x >> 3;
        slice = rest % NS;
        vh = (rest / NS) * 8 + x;
        if (vh >= a.B * a.Hq) return;
    }
    const bool writes_out = a.out != nullptr && a.mode != MODE_PREFILL;
    if (slice != 0 && !writes_out) return;
    // Virtual head vh = u * B * Hq + bh: query position u of head bh (u = 0 unless
    // a batched prefill launch); the workspaces are indexed by vh, the cache, q
    // and the outputs by bh.
    const int u = kMulti ? vh / (a.B * a.Hq) : 0;
    const int bh = kMulti ? vh - u * a.B * a.Hq : vh;
    const int64_t len = kMulti ? a.len + u : a.len;

    if (slice == 0 && (a.mode == MODE_REFRESH || a.mode == MODE_COLD)) {
        const int8_t code = a.mode == MODE_REFRESH ? PATH_REFRESH : PATH_COLD;
        if (tid == 0) {
            if (a.dbg_path) a.dbg_path[bh] = code;
            if (a.dbg_rho) a.dbg_rho[bh] = __builtin_nan("");
        }
        if (a.dbg_ret)
            for (int i = tid; i < a.R; i += NT) a.dbg_ret[(int64_t)bh * a.R + i] = -1;
    }
    if constexpr (!kMulti) {
        if (writes_out && final_fast<T, D, NS, EPT>(a, w, bh, slice, fs, sm.ent, sm.sel, s_part))
            return;
        __syncthreads();   // the general path follows the fast path's early exit
    }

    // Path, the region counts of both layouts and the first entries of every
    // region in one round trip (the entry loads are speculative: a region's
    // count is known only afterwards).
    const bool sel_mode = a.mode == MODE_SELECT;
    const int8_t path_g = sel_mode ? w.path[bh] : (int8_t)PATH_FALLBACK;
    const bool reuse = path_g == PATH_REUSE || path_g == PATH_REUSE_SCANNED;
    const int nreg_s = (int)((len + kFilterRows - 1) / kFilterRows);
    const int rpt = (nreg_s + NT - 1) / NT;
    uint32_t scnt[kRegPerThread];
#pragma unroll
    for (int u = 0; u < kRegPerThread; ++u) {
        const int r = tid * rpt + u;
        const bool ok = u < rpt && r < nreg_s;
        const uint32_t x = w.surv_cnt[(int64_t)vh * a.n_regions + (ok ? r : 0)];
        scnt[u] = ok ? x : 0u;
    }
    const uint32_t ccnt_l = w.cand_cnt[(int64_t)bh * kCandRanges + (tid < kCandRanges ? tid : 0)];
    const uint32_t ccnt = (sel_mode && tid < kCandRanges) ? ccnt_l : 0u;

    Regions rg;
    if (reuse) {
        rg.base = w.cand_ent + (int64_t)bh * kCandRanges * a.cand_cap;
        rg.stride = a.cand_cap;
        rg.nreg = kCandRanges;
    } else {
        rg.base = w.surv + (int64_t)vh * a.row_stride;
        rg.stride = kFilterRows;
        rg.nreg = nreg_s;
    }
    // spec slots per region: kSpecLoads * NT spread over the regions
    int spec = (kSpecLoads * NT) / rg.nreg;
    spec = spec < (int)rg.stride ? spec : (int)rg.stride;
    uint64_t sv[kSpecLoads];
#pragma unroll
    for (int u = 0; u < kSpecLoads; ++u) {
        const int e = tid + u * NT;
        const int r = spec > 0 && e < spec * rg.nreg ? e / spec : 0;
        const int j = spec > 0 && e < spec * rg.nreg ? e - r * spec : 0;
        sv[u] = rg.base[(int64_t)r * rg.stride + j];
    }
    for (int i = tid; i < kHistBins; i += NT) sm.hist[i] = 0u;
    if (tid == 0) {
        sm.rmax = 0ull;
        sm.rmin = ~0ull;
        sm.n_tie = 0u;
        sm.thr = 0ull;
    }
    {
        uint32_t mine = 0;
        if (reuse) {
            mine = ccnt;
        } else {
#pragma unroll
            for (int u = 0; u < kRegPerThread; ++u) mine += scnt[u];
        }
        uint32_t total;
        uint32_t run = block_excl_scan<NT>(mine, sm.redu, &total);
        if (reuse) {
            if (tid < kCandRanges) sm.pref[tid] = run;
        } else {
#pragma unroll
            for (int u = 0; u < kRegPerThread; ++u) {
                const int r = tid * rpt + u;
                if (u < rpt && r < nreg_s) {
                    sm.pref[r] = run;
                    run += scnt[u];
                }
            }
        }
        if (tid == 0) sm.pref[rg.nreg] = total;
        __syncthreads();
        rg.n = (int)total;
    }
    rg.pref = sm.pref;
    rg.staged = nullptr;
    rg.top = rg.nreg > 1 ? 1 << (31 - __clz(rg.nreg - 1)) : 0;
    {
        // Stage the entries in index order (when they fit) and find the largest
        // and smallest rank.
        uint64_t lmax = 0ull, lmin = ~0ull;
        if (rg.n <= kEntCache) {
#pragma unroll
            for (int u = 0; u < kSpecLoads; ++u) {
                const int e = tid + u * NT;
                if (spec > 0 && e < spec * rg.nreg) {
                    const int r = e / spec, j = e - r * spec;
                    const int at = (int)sm.pref[r] + j;
                    if (at < (int)sm.pref[r + 1]) {
                        sm.ent[at] = sv[u];
                        lmax = sv[u] > lmax ? sv[u] : lmax;
                        lmin = sv[u] < lmin ? sv[u] : lmin;
                    }
                }
            }
            // entries past the speculative slots: one wave per region
            for (int r = wave; r < rg.nreg; r += NW) {
                const int p0 = (int)sm.pref[r], c = (int)sm.pref[r + 1] - p0;
                for (int j0 = spec; j0 < c; j0 += 4 * 64) {
                    uint64_t e[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int j = j0 + u * 64 + lane;
                        e[u] = rg.base[(int64_t)r * rg.stride + (j < c ? j : 0)];
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int j = j0 + u * 64 + lane;
                        if (j < c) {
                            sm.ent[p0 + j] = e[u];
                            lmax = e[u] > lmax ? e[u] : lmax;
                            lmin = e[u] < lmin ? e[u] : lmin;
                        }
                    }
                }
            }
        } else {
            for (int j0 = 0; j0 < rg.n; j0 += 4 * NT) {
                uint64_t e[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int j = j0 + u * NT + tid;
                    e[u] = rg.get(j < rg.n ? j : 0);
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int j = j0 + u * NT + tid;
                    if (j < rg.n) {
                        lmax = e[u] > lmax ? e[u] : lmax;
                        lmin = e[u] < lmin ? e[u] : lmin;
                    }
                }
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const uint64_t omax = __shfl_xor((unsigned long long)lmax, o);
            const uint64_t omin = __shfl_xor((unsigned long long)lmin, o);
            lmax = omax > lmax ? omax : lmax;
            lmin = omin < lmin ? omin : lmin;
        }
        if (lane == 0) {
            atomicMax(&sm.rmax, (unsigned long long)lmax);
            atomicMin(&sm.rmin, (unsigned long long)lmin);
        }
        __syncthreads();
        if (rg.n <= kEntCache) rg.staged = sm.ent;
    }

    // Top-K (Eq. 1 / Eq. 11): the entries e >= thr; then those in index order.
    uint64_t thr = 0ull;
    if (rg.n > a.K) {
        bool done = false;
        if (rg.staged) done = value_threshold<FinalSmem<D, DS, NT>, NT>(rg.staged, rg.n, a.K, sm, thr);
        if (!done) {
            uint64_t prefix, mask;
            radix_threshold<FinalSmem<D, DS, NT>, NT>(rg, a.K, sm, prefix, mask);
            thr = mask == 0ull ? 0ull : prefix;
        }
    }
    const int kn = rg.n < a.K ? rg.n : a.K;
    {
        // Wave w compacts entries [w * per, (w + 1) * per) in order, 64 consecutive
        // entries per ballot (conflict-free LDS reads): one pass counts its
        // selected entries, a second writes them after those of the waves before.
        const int per = ((rg.n + NW - 1) / NW + 63) & ~63;
        const int jb = wave * per, je = min(jb + per, rg.n);
        const uint64_t below = (1ull << lane) - 1ull;
        const uint64_t *stg = rg.staged;
        // staged entries are read from LDS directly (no per-entry branch)
        auto entry = [&](int j) { return stg ? stg[j] : rg.get(j); };
        uint32_t cnt = 0u;
        for (int j0 = jb; j0 < je; j0 += 4 * 64) {
            uint64_t e[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int j = j0 + u * 64 + lane;
                e[u] = entry(j < je ? j : jb);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                cnt += (uint32_t)__popcll(__ballot(j0 + u * 64 + lane < je && e[u] >= thr));
        }
        if (lane == 0) sm.wcnt[wave] = cnt;
        __syncthreads();
        uint32_t pos = 0u;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) pos += ww < wave ? sm.wcnt[ww] : 0u;
        for (int j0 = jb; j0 < je; j0 += 4 * 64) {
            uint64_t e[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int j = j0 + u * 64 + lane;
                e[u] = entry(j < je ? j : jb);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool s = j0 + u * 64 + lane < je && e[u] >= thr;
                const uint64_t bal = __ballot(s);
                const uint32_t at = pos + (uint32_t)__popcll(bal & below);
                if (s && at < (uint32_t)kMaxK)
                    sm.sel[at] = ((uint64_t)rank_index(e[u]) << 32) | rank_key(e[u]);
                pos += (uint32_t)__popcll(bal);
            }
        }
        __syncthreads();
    }

    if (writes_out) {
        // Eq. 12 on this block's slice of the head dimension; the largest selected
        // score is the top rank's.
        const float mx = key_score(rank_key((uint64_t)sm.rmax));
        const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;
        const T *vbase = (const T *)a.v + ((int64_t)b * a.Hkv + g) * a.max_len * D + slice * DS;
        const int sub = lane / LPR, vl = lane % LPR;
        float acc[EPV];
#pragma unroll
        for (int e = 0; e < EPV; ++e) acc[e] = 0.0f;
        float lsum = 0.0f;
#pragma unroll 4
        for (int t = wave * RPW + sub; t < kn; t += NW * RPW) {
            const uint64_t se = sm.sel[t];
            const uint4 raw = ((const uint4 *)(vbase + (int64_t)(uint32_t)(se >> 32) * D))[vl];
            const float wt = expf(key_score((uint32_t)se) - mx);
            Dot<T>::axpy(raw, wt, acc);
            lsum += vl == 0 ? wt : 0.0f;
        }
#pragma unroll
        for (int o = LPR; o < 64; o <<= 1) {
#pragma unroll
            for (int e = 0; e < EPV; ++e) acc[e] += __shfl_xor(acc[e], o);
            lsum += __shfl_xor(lsum, o);
        }
        if (sub == 0) {
#pragma unroll
            for (int e = 0; e < EPV; ++e) sm.part[wave][vl * EPV + e] = acc[e];
            if (vl == 0) sm.lpart[wave] = lsum;
        }
        __syncthreads();
        if (tid < DS) {
            float o = 0.0f, l = 0.0f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) {
                o += sm.part[ww][tid];
                l += sm.lpart[ww];
            }
            a.out[(int64_t)bh * D + slice * DS + tid] = kn > 0 ? o / l : 0.0f;
        }
    }
    // The writes that follow are shared out over the head's blocks, each of which
    // holds the whole selection in LDS: the support output, the cache entry's
    // support and count, its q_bar, and the counters or the histogram reset.
    const int nblk = writes_out ? NS : 1;
    auto owns = [&](int job) { return job % nblk == slice; };
    if (owns(0)) {
        if (writes_out && a.sel != nullptr)
            for (int t = tid; t < a.K; t += NT)
                a.sel[(int64_t)bh * a.K + t] = t < kn ? (int32_t)(sm.sel[t] >> 32) : -1;
        if (a.dbg_ncand && tid == 0) a.dbg_ncand[bh] = reuse ? rg.n : 0;
        if (a.dbg_cand)
            for (int j = tid; j < a.cand_cap; j += NT)
                a.dbg_cand[(int64_t)bh * a.cand_cap + j] = (reuse && j < rg.n) ? (int32_t)rank_index(rg.get(j)) : -1;
    }
    if (a.do_insert) {
        // Sec. 3.4: insert (q_bar, support) after either path.
        const int64_t e = (int64_t)bh * a.M + (kMulti ? (a.insert_slot + u) % a.M : a.insert_slot);
        if (owns(1)) {
            for (int t = tid; t < a.K; t += NT)
                w.supp[e * a.K + t] = t < kn ? (int32_t)(sm.sel[t] >> 32) : -1;
            if (tid == 0) w.cnt[e] = kn;
        }
        if (owns(2)) {
            if (a.mode == MODE_SELECT) {
                for (int t = tid; t < D; t += NT) w.qbar[e * D + t] = w.qbar_cur[(int64_t)bh * D + t];
            } else {
                const T *q = (const T *)a.q + (int64_t)bh * a.q_head_stride + (int64_t)u * D;
                block_qbar<T, D, NT>(q, sm.qbar, sm.red64);
                for (int t = tid; t < D; t += NT) w.qbar[e * D + t] = sm.qbar[t];
            }
        }
    }
    if (owns(3)) {
        if (reuse) {
            if (tid == 0) {
                atomicAdd(&w.stats[STAT_CAND_SUM], (unsigned long long)rg.n);
                atomicMax(&w.stats[STAT_CAND_MAX], (unsigned long long)rg.n);
            }
        } else {
            // leave the histogram zeroed for the next launch
            for (int i = tid; i < kHistBins; i += NT) w.hist[(int64_t)vh * kHistBins + i] = 0u;
        }
    }
}

// ---------------------------------------------------------------------------
// Batched prefill initialisation (Sec. 3.3): the prompt-tail queries of U
// positions at once, each against its causal prefix
// ---------------------------------------------------------------------------


// k_pf_score: the scores of Eq. 4 for U positions x G heads of a KV group (the
// group's "virtual queries", vq = u * G + j) as a matrix product on the matrix
// cores.  Block (pair, tile) takes keys [kc * kPfKeys, ...) of KV group grp for
// the kPfCols virtual queries of query tile `tile`, in column tiles of 16, with
// v_mfma_f32_16x16x32_bf16: the A operand is 16 key rows x 32 dims, B is 32 dims
// x 16 queries, and lane l supplies key row (and query) l % 16 for dims
// 8 (l / 16) .. + 7 of each 32-dim step and receives keys 4 (l / 16) .. + 3 of
// query l % 16.  Each key tile loaded serves every column tile.  Keys at or past
// a query's causal length are left out of its histogram (LDS, two 16-bit counts
// per word, added to the global histogram at the end); every score is stored to
// the virtual head's score row, those past the causal length included (no later
// stage reads them), so that each wave issues the same stores every iteration
// and its key loads, two iterations ahead, never wait for them.  The blocks of
// one (group, key chunk) pair share blockIdx % 8, so they run on one XCD and
// read the chunk's keys through one L2.
template <int D>
__global__ __launch_bounds__(kPfThreads) void k_pf_score(StepArgs a, Ws w, Geometry geo)
{
    constexpr int NT = kPfThreads, NW = NT / 64, TW = kPfTiles, KS = D / 32;
    constexpr int CT = kPfCols / 16;
    constexpr int ROWS = NW * TW * 16;
    constexpr int ITERS = kPfKeys / ROWS;
    // A chunk's stores stay inside its score row: chunks end on filter-region
    // boundaries, and score rows are whole regions long.
    static_assert(D % 32 == 0 && kPfKeys % (2 * ROWS) == 0 && kFilterRows % kPfKeys == 0 &&
                  kPfCols % 16 == 0, "tile geometry");
    static_assert(kPfKeys < 65536 && kPfHistStride * 2 > kHistBins, "16-bit bin counts");
    __shared__ uint32_t s_hist[kPfCols * kPfHistStride];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, kq = lane >> 4;
    const int j = (int)blockIdx.x;
    const int pair = (j & 7) + 8 * (j / (8 * geo.pf_qtiles));
    const int tile = (j >> 3) % geo.pf_qtiles;
    if (pair >= geo.pf_pairs) return;
    const int grp = pair / geo.pf_kchunks, kc = pair % geo.pf_kchunks;
    const int b = grp / a.Hkv, g = grp % a.Hkv;
    const int BH = a.B * a.Hq;
    const int nvq = a.G * a.U;
    // rows of this block: the chunk, cut at the longest causal length of the tile
    const int last_vq = (tile + 1) * kPfCols - 1 < nvq - 1 ? (tile + 1) * kPfCols - 1 : nvq - 1;
    const int64_t tlen = a.len + last_vq / a.G;
    const int64_t k0 = (int64_t)kc * kPfKeys;
    const int64_t k1 = k0 + kPfKeys < tlen ? k0 + kPfKeys : tlen;
    if (k0 >= k1) return;

    // This lane's virtual query in each column tile; columns past the last one
    // repeat it (same query, same score row, same values stored) and count nothing.
    bf16x8_t qb[CT][KS];
    float *srow[CT];
    int64_t cend[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
        const int vq = tile * kPfCols + ct * 16 + col;
        const bool cvalid = vq < nvq;
        const int vqe = cvalid ? vq : nvq - 1;
        const int u = vqe / a.G;
        const int bh = b * a.Hq + g * a.G + vqe % a.G;
        const uint4 *qr = (const uint4 *)((const uint16_t *)a.q + (int64_t)bh * a.q_head_stride +
                                          (int64_t)u * D);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qb[ct][ks] = __builtin_bit_cast(bf16x8_t, qr[ks * 4 + kq]);
        srow[ct] = w.scores + ((int64_t)u * BH + bh) * a.row_stride;
        const int64_t clen = cvalid ? a.len + u : 0;
        cend[ct] = clen < k1 ? clen : k1;           // rows counted for this query
    }
    const uint16_t *kbase = (const uint16_t *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    auto load = [&](uint4 (&kv)[TW][KS], int64_t base) {
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            const int64_t r = base + (wave * TW + t) * 16 + col;
            const uint4 *rp = (const uint4 *)(kbase + (r < k1 ? r : k0) * D);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kv[t][ks] = rp[ks * 4 + kq];
        }
    };
    // One iteration: the scores of ROWS keys from kv, the loads of the keys two
    // iterations on into kv, the stores and the histogram counts.
    auto step = [&](uint4 (&kv)[TW][KS], int64_t base) {
        f32x4_t acc[CT][TW];
#pragma unroll
        for (int t = 0; t < TW; ++t)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                acc[ct][t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    acc[ct][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8_t, kv[t][ks]), qb[ct][ks], acc[ct][t], 0, 0, 0);
            }
        load(kv, base + 2 * ROWS);   // past k1 the clamped rows are re-read, never used
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            uint32_t *hrow = s_hist + (ct * 16 + col) * kPfHistStride;
#pragma unroll
            for (int t = 0; t < TW; ++t) {
                const int64_t r4 = base + (wave * TW + t) * 16 + 4 * kq;
                const float sc[4] = {acc[ct][t][0] * a.inv_sqrt_d, acc[ct][t][1] * a.inv_sqrt_d,
                                     acc[ct][t][2] * a.inv_sqrt_d, acc[ct][t][3] * a.inv_sqrt_d};
                *(float4 *)(srow[ct] + r4) = make_float4(sc[0], sc[1], sc[2], sc[3]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (r4 + i < cend[ct]) {
                        const uint32_t bin = ord_key(sc[i]) >> kHistShift;
                        atomicAdd(&hrow[bin >> 1], 1u << ((bin & 1u) << 4));
                    }
                }
            }
        }
    };
    uint4 kva[TW][KS], kvb[TW][KS];
    load(kva, k0);   // the first key rows are in flight while the histogram is cleared
    load(kvb, k0 + ROWS);
    for (int i = tid; i < kPfCols * kPfHistStride; i += NT) s_hist[i] = 0u;
    __syncthreads();
    // A fixed trip count: rows past k1 (the chunk cut short by the causal limit)
    // are computed from clamped loads and stored where nothing reads them.
    for (int it = 0; it < ITERS; it += 2) {
        step(kva, k0 + (int64_t)it * ROWS);
        step(kvb, k0 + (int64_t)(it + 1) * ROWS);
    }
    __syncthreads();
    for (int i = tid; i < kPfCols * kHistBins; i += NT) {
        const int c = i / kHistBins, bin = i % kHistBins;
        const int cvq = tile * kPfCols + c;
        const uint32_t n = (s_hist[c * kPfHistStride + (bin >> 1)] >> ((bin & 1) << 4)) & 0xFFFFu;
        if (n && cvq < nvq) {
            const int cbh = b * a.Hq + g * a.G + cvq % a.G;
            atomicAdd(&w.hist[((int64_t)(cvq / a.G) * BH + cbh) * kHistBins + bin], n);
        }
    }
}

// ---------------------------------------------------------------------------
// Full attention (the dense baseline): softmax over every row, then V
// ---------------------------------------------------------------------------

// k_dense: block (b, g, c) takes rows [c * kDenseRows, ...) of KV group (b, g) for
// the G query heads of the group (one key or value row load serves all of them):
// scores with the scan's row geometry, then per head the chunk's maximum m, the
// weights exp(s - m), their sum l and the weighted sum o of the value rows.
// (o, m, l) go to dense_part; k_dense_merge rescales and adds the chunks.
template <typename T, int D, int G>
__global__ __launch_bounds__(kDenseThreads, (kDenseWaves<T, D, G>)) void k_dense(StepArgs a, Ws w)
{
    using R = RowT<T, D>;
    constexpr int NT = kDenseThreads, NW = NT / 64;
    constexpr int VL = D * (int)sizeof(T) / 16;     // lanes per value row (16 bytes each)
    constexpr int VR = 64 / VL;                      // value rows per wave instruction
    constexpr int EPV = 16 / (int)sizeof(T);
    static_assert(VL >= 1 && VL <= 64 && 64 % VL == 0, "value row geometry");
    __shared__ float s_sc[G][kDenseRows];
    __shared__ float s_red[NW][G];
    __shared__ float s_ml[2][G];            // each head's chunk maximum and weight sum
    __shared__ float s_o[NW][G][D];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int nch = (int)((a.len + kDenseRows - 1) / kDenseRows);
    const int c = blockIdx.x % nch, bg = blockIdx.x / nch;
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    const int bh0 = b * a.Hq + g * a.G;      // heads past a.G pad the group
    const int64_t r0 = (int64_t)c * kDenseRows;
    const int nrow = (int)(a.len - r0 < kDenseRows ? a.len - r0 : kDenseRows);
    const T *kbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    const T *vbase = (const T *)a.v + ((int64_t)b * a.Hkv + g) * a.max_len * D;

    if constexpr (G == 8) {
        // scores (Eq. 4) of the chunk's rows in the octet layout of
        // scan_segment_octet: lane o owns head o's score of its row
        constexpr int NV = R::kBytes / 128, RPP = NT / 8, UP = 2 * kScanRowsPerIter / RPP;
        const int o = tid & 7, rr = tid >> 3;
        uint4 qv[G][NV];
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int hj = j < a.G ? j : 0;
            const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)(bh0 + hj) * a.q_head_stride);
#pragma unroll
            for (int v = 0; v < NV; ++v) qv[j][v] = qr[v * 8 + o];
        }
        for (int base = 0; base < nrow; base += UP * RPP) {
            uint4 kv[UP][NV];
            int row[UP];
#pragma unroll
            for (int u = 0; u < UP; ++u) {
                row[u] = base + u * RPP + rr;
                const uint4 *rp = (const uint4 *)(kbase + (r0 + (row[u] < nrow ? row[u] : 0)) * D);
#pragma unroll
                for (int v = 0; v < NV; ++v) kv[u][v] = rp[v * 8 + o];
            }
#pragma unroll
            for (int u = 0; u < UP; ++u) {
                float acc[G];
#pragma unroll
                for (int j = 0; j < G; ++j) {
                    float s0 = 0.0f;
#pragma unroll
                    for (int v = 0; v < NV; ++v) s0 = Dot<T>::f(kv[u][v], qv[j][v], s0);
                    acc[j] = s0;
                }
                const float sc = octet_transpose_sum(acc, o) * a.inv_sqrt_d;
                if (row[u] < nrow) s_sc[o][row[u]] = sc;
            }
        }
    } else {
    uint4 qv[G][R::kNV];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const int hj = j < a.G ? j : 0;
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)(bh0 + hj) * a.q_head_stride);
#pragma unroll
        for (int v = 0; v < R::kNV; ++v) qv[j][v] = qr[v * 4 + p];
    }
    // scores (Eq. 4) of the chunk's rows, two rows per lane per pass
    for (int base = 0; base < nrow; base += 2 * kScanRowsPerIter) {
        uint4 kv[2][R::kNV];
        int row[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            row[u] = base + u * kScanRowsPerIter + wave * 16 + rl;
            const uint4 *rp = (const uint4 *)(kbase + (r0 + (row[u] < nrow ? row[u] : 0)) * D);
#pragma unroll
            for (int v = 0; v < R::kNV; ++v) kv[u][v] = rp[v * 4 + p];
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            float acc[G];
#pragma unroll
            for (int j = 0; j < G; ++j) {
                float s0 = 0.0f;
#pragma unroll
                for (int v = 0; v < R::kNV; ++v) s0 = Dot<T>::f(kv[u][v], qv[j][v], s0);
                acc[j] = s0;
            }
            float sc_lo, sc_hi;
            group_scores<G>(acc, p, sc_lo, sc_hi);
            if (row[u] < nrow) {
#pragma unroll
                for (int jj = 0; jj < (G + 3) / 4; ++jj) {
                    const int j = jj * 4 + (G == 1 ? 0 : (G == 2 ? (p & 1) : p));
                    const bool mine = G == 1 ? p == 0 : (G == 2 ? p < 2 : true);
                    if (mine) s_sc[j][row[u]] = (jj == 0 ? sc_lo : sc_hi) * a.inv_sqrt_d;
                }
            }
        }
    }
    }
    __syncthreads();
    // per head: chunk maximum, then weights exp(s - m) in place and their sum
    float m[G], l[G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        float x = -INFINITY;
        for (int i = tid; i < nrow; i += NT) x = fmaxf(x, s_sc[j][i]);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
        if (lane == 0) s_red[wave][j] = x;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < G; ++j) {
        m[j] = s_red[0][j];
#pragma unroll
        for (int i = 1; i < NW; ++i) m[j] = fmaxf(m[j], s_red[i][j]);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < G; ++j) {
        float x = 0.0f;
        for (int i = tid; i < nrow; i += NT) {
            const float e = expf(s_sc[j][i] - m[j]);
            s_sc[j][i] = e;
            x += e;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
        if (lane == 0) s_red[wave][j] = x;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < G; ++j) {
        l[j] = 0.0f;
#pragma unroll
        for (int i = 0; i < NW; ++i) l[j] += s_red[i][j];
    }
    if (tid == 0) {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            s_ml[0][j] = m[j];
            s_ml[1][j] = l[j];
        }
    }
    // Eq. 12 over the chunk: VL lanes per value row, each holding EPV elements
    // for every head; rows spread over the waves (VU rows per lane in flight).
    constexpr int VU = G == 8 ? 2 : 4;
    const int sub = lane / VL, vl = lane % VL;
    float acc[G][EPV];
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
        for (int e = 0; e < EPV; ++e) acc[j][e] = 0.0f;
    for (int t0 = wave * VR; t0 < nrow; t0 += NW * VR * VU) {
        uint4 raw[VU];
#pragma unroll
        for (int u = 0; u < VU; ++u) {
            const int t = t0 + u * NW * VR + sub;
            raw[u] = ((const uint4 *)(vbase + (r0 + (t < nrow ? t : 0)) * D))[vl];
        }
#pragma unroll
        for (int u = 0; u < VU; ++u) {
            const int t = t0 + u * NW * VR + sub;
            if (t < nrow) {
#pragma unroll
                for (int j = 0; j < G; ++j) Dot<T>::axpy(raw[u], s_sc[j][t], acc[j]);
            }
        }
    }
#pragma unroll
    for (int o = VL; o < 64; o <<= 1)
#pragma unroll
        for (int j = 0; j < G; ++j)
#pragma unroll
            for (int e = 0; e < EPV; ++e) acc[j][e] += __shfl_xor(acc[j][e], o);
    if (sub == 0)
#pragma unroll
        for (int j = 0; j < G; ++j)
#pragma unroll
            for (int e = 0; e < EPV; ++e) s_o[wave][j][vl * EPV + e] = acc[j][e];
    __syncthreads();
    for (int i = tid; i < a.G * D; i += NT) {
        const int j = i / D, e = i % D;
        float o = 0.0f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) o += s_o[ww][j][e];
        float *dst = w.dense_part + ((int64_t)(bh0 + j) * a.n_dense + c) * (D + 2);
        dst[e] = o;
        if (e == 0) {
            dst[D] = s_ml[0][j];
            dst[D + 1] = s_ml[1][j];
        }
    }
}

// k_dense_merge: one block per head; out = sum_c e^(m_c - M) o_c / sum_c e^(m_c - M) l_c
// with M the largest chunk maximum.  Each wave folds its share of the chunks
// into a running (maximum, sum, output) with rescaling, so every chunk is read
// once, all in one round trip; the waves' partials are then combined the same way.
template <int D>
__global__ __launch_bounds__(kMergeThreads) void k_dense_merge(StepArgs a, Ws w)
{
    constexpr int NT = kMergeThreads, NW = NT / 64, EPL = D / 64, U = 8;
    static_assert(D % 64 == 0, "whole elements per lane");
    __shared__ float s_m[NW], s_l[NW];
    __shared__ float s_o[NW][D];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, bh = blockIdx.x;
    const int nch = (int)((a.len + kDenseRows - 1) / kDenseRows);
    const float *part = w.dense_part + (int64_t)bh * a.n_dense * (D + 2);
    float mw = -INFINITY, lw = 0.0f, acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.0f;
    for (int c0 = wave; c0 < nch; c0 += NW * U) {
        float mv[U], lv[U], ov[U][EPL];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * NW < nch ? c0 + u * NW : c0;
            const float *pc = part + (int64_t)c * (D + 2);
            mv[u] = pc[D];
            lv[u] = pc[D + 1];
#pragma unroll
            for (int e = 0; e < EPL; ++e) ov[u][e] = pc[lane * EPL + e];
        }
        float mn = mw;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c0 + u * NW < nch) mn = fmaxf(mn, mv[u]);
        const float f0 = mw == -INFINITY ? 0.0f : expf(mw - mn);
        lw *= f0;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] *= f0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float f = c0 + u * NW < nch ? expf(mv[u] - mn) : 0.0f;
            lw += f * lv[u];
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[e] += f * ov[u][e];
        }
        mw = mn;
    }
    if (lane == 0) {
        s_m[wave] = mw;
        s_l[wave] = lw;
    }
#pragma unroll
    for (int e = 0; e < EPL; ++e) s_o[wave][lane * EPL + e] = acc[e];
    __syncthreads();
    if (tid < D) {
        float M = -INFINITY;
#pragma unroll
        for (int i = 0; i < NW; ++i) M = fmaxf(M, s_m[i]);
        float L = 0.0f, o = 0.0f;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const float f = s_m[i] == -INFINITY ? 0.0f : expf(s_m[i] - M);
            L += f * s_l[i];
            o += f * s_o[i][tid];
        }
        a.out[(int64_t)bh * D + tid] = o / L;
    }
}

// ---------------------------------------------------------------------------
// k_scan_list: the full-history scan of every KV group (exact, refresh and cold
// steps) when the groups' whole filter regions of kFilterRows rows give every
// CU at least one.  One block per whole region keeps the region's scores in
// LDS and writes only the entries in the bins at or above the one holding the
// region's own K-th largest score, as ranks in index order (the region's local
// survivors), with their count in surv_cnt.  The rows past the last whole
// region of a group are shared out over the group's blocks, which write those
// scores to the score row as the score-row scan does.  k_filter then keeps the
// entries at or above the head's threshold bin b* (Eq. 1 through the
// histogram): a block's rows are a subset of the head's, so at least K of the
// head's rows lie in bins at or above the block's local bin, b* is never below
// it, and the global survivors are exactly those the score-row path compacts.
// For the same reason a block adds to the head's histogram only its counts of
// the bins from its local bin up: the counts k_filter sums from the top down to
// b* are complete, and it reads no lower bin.
// One block per CU (its LDS holds the region's scores and histograms): 1024
// threads where the group's query vectors and two key rows a lane fit in 128
// registers, else 512 threads with up to 256; each lane keeps the next pass's
// key rows in flight while it scores the current ones.
// ---------------------------------------------------------------------------

__host__ __device__ constexpr int scan_list_lds(int g) { return g * (kFilterRows + kHistBins) * 4; }

template <typename T, int D, int G>
constexpr int kListThreads = (G + 2) * RowT<T, D>::kNV * 4 <= 96 ? 1024 : 512;
template <typename T, int D, int G>
constexpr int kListRowsInFlight = kListThreads<T, D, G> == 1024 ? 1 : ((G + 4) * RowT<T, D>::kNV * 4 <= 192 ? 2 : 1);

template <typename T, int D, int G>
__global__ __launch_bounds__((kListThreads<T, D, G>), (kListThreads<T, D, G> / 256)) void k_scan_list(StepArgs a, Ws w)
{
    using R = RowT<T, D>;
    constexpr int NT = kListThreads<T, D, G>, NW = NT / 64;
    constexpr int U = kListRowsInFlight<T, D, G>;       // rows per lane per pass
    constexpr int RPP = NT / 4;                          // rows per pass and row slot
    constexpr int STEP = U * RPP;                        // rows per pass
    constexpr int WPH = NW / G;                          // compaction waves per head
    constexpr int RPL = kFilterRows / (WPH * 64);        // compaction rows per lane
    static_assert(G == 1 || G == 2 || G == 4, "quad row layout");
    static_assert(kFilterRows % (2 * STEP) == 0 && RPL % 4 == 0 && RPL <= 32, "region geometry");
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    float *s_sc = (float *)lds;                                       // [G][kFilterRows]
    uint32_t *s_hist = (uint32_t *)(lds + G * kFilterRows * 4);       // [G][kHistBins]
    __shared__ uint32_t s_bloc[G];
    __shared__ uint32_t s_wcnt[NW];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, p = lane & 3, rl = lane >> 2;
    const int nfull = (int)(a.len / kFilterRows);        // whole regions per group (>= 1)
    const int gi = (int)blockIdx.x / nfull, f = (int)blockIdx.x - gi * nfull;
    const int b = gi / a.Hkv, g = gi % a.Hkv;
    const int bh0 = b * a.Hq + g * a.G;
    const int64_t r0 = (int64_t)f * kFilterRows;
    const T *gbase = (const T *)a.k + ((int64_t)b * a.Hkv + g) * a.max_len * D;
    const T *kbase = gbase + r0 * D;
    // this block's share of the rows past the last whole region: [x0, x1)
    const int64_t tail0 = (int64_t)nfull * kFilterRows;
    const int64_t xs = ((a.len - tail0) + nfull - 1) / nfull;
    const int64_t x0 = tail0 + f * xs < a.len ? tail0 + f * xs : a.len;
    const int64_t x1 = x0 + xs < a.len ? x0 + xs : a.len;

    uint4 qv[G][R::kNV];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const int hj = j < a.G ? j : 0;   // heads past a.G pad the group
        const uint4 *qr = (const uint4 *)((const T *)a.q + (int64_t)(bh0 + hj) * a.q_head_stride);
#pragma unroll
        for (int v = 0; v < R::kNV; ++v) qv[j][v] = qr[v * 4 + p];
    }
    // Key rows base + u * RPP + wave * 16 + rl of a pass, from clamped (in-bounds)
    // rows; two register sets, so that a pass's loads are issued before the
    // previous pass is scored.
    uint4 kA[U][R::kNV], kB[U][R::kNV];
    auto load = [&](uint4 (&kv)[U][R::kNV], const T *src, int base, int n) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = base + u * RPP + wave * 16 + rl;
            const uint4 *rp = (const uint4 *)(src + (int64_t)(r < n ? r : 0) * D);
#pragma unroll
            for (int v = 0; v < R::kNV; ++v) kv[u][v] = rp[v * 4 + p];
        }
    };
    // Scores of a pass: to LDS (the region) or to the score row (rows past the
    // last whole region), counted in the block's histograms either way.
    auto score = [&](const uint4 (&kv)[U][R::kNV], int base, int n, float *row_out) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = base + u * RPP + wave * 16 + rl;
            float acc[G];
#pragma unroll
            for (int j = 0; j < G; ++j) {
                float s0 = 0.0f;
#pragma unroll
                for (int v = 0; v < R::kNV; ++v) s0 = Dot<T>::f(kv[u][v], qv[j][v], s0);
                acc[j] = s0;
            }
            float sc_lo, sc_hi;
            group_scores<G>(acc, p, sc_lo, sc_hi);
            const int j = G == 1 ? 0 : (G == 2 ? (p & 1) : p);
            const bool mine = G == 1 ? p == 0 : (G == 2 ? p < 2 : true);
            if (mine && j < a.G && r < n) {
                const float sc = sc_lo * a.inv_sqrt_d;
                if (row_out) row_out[(int64_t)j * a.row_stride + r] = sc;
                else s_sc[j * kFilterRows + r] = sc;
                atomicAdd(&s_hist[j * kHistBins + (ord_key(sc) >> kHistShift)], 1u);
            }
        }
    };
    load(kA, kbase, 0, kFilterRows);   // the first rows are in flight while the histogram is cleared
    for (int i = tid; i < G * kHistBins; i += NT) s_hist[i] = 0u;
    __syncthreads();
    for (int base = 0; base < kFilterRows; base += 2 * STEP) {
        load(kB, kbase, base + STEP, kFilterRows);
        score(kA, base, kFilterRows, nullptr);
        if (base + 2 * STEP < kFilterRows) load(kA, kbase, base + 2 * STEP, kFilterRows);
        score(kB, base + STEP, kFilterRows, nullptr);
    }
    if (x1 > x0) {
        const int nx = (int)(x1 - x0);
        float *row_out = w.scores + (int64_t)bh0 * a.row_stride + x0;
        for (int base = 0; base < nx; base += STEP) {
            load(kA, gbase + x0 * D, base, nx);
            score(kA, base, nx, row_out);
        }
    }
    __syncthreads();

    // Wave j: the bin holding head j's K-th largest score of the block.  Lane l
    // reads the 4-bin groups l + 64 i (i = 0..7: chunk i holds bins 256 i ..
    // 256 i + 255), so that the wave's reads are contiguous; the chunk totals
    // locate the chunk, a suffix sum over the lanes the group, the lane the bin.
    // The lanes keep their counts for the histogram flush at the end (no barrier
    // then waits for those atomics).
    uint32_t c[8][4];
    uint32_t bloc = 0u;
    if (wave < a.G) {
        const uint4 *hv = (const uint4 *)(s_hist + wave * kHistBins);
        uint32_t cs[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint4 x = hv[i * 64 + lane];
            c[i][0] = x.x;
            c[i][1] = x.y;
            c[i][2] = x.z;
            c[i][3] = x.w;
            cs[i] = x.x + x.y + x.z + x.w;
        }
        const uint32_t kn = (uint32_t)a.K;              // <= kFilterRows rows counted
        uint32_t above = 0u, ic = 0u;
        bool found = false;
#pragma unroll
        for (int i = 7; i >= 0; --i) {
            const uint32_t t = wave_incl_scan(cs[i]);
            const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)t, 63);
            if (!found && above + tot >= kn) {
                found = true;
                ic = (uint32_t)i;
            } else if (!found) {
                above += tot;
            }
        }
        // chunk ic: lane l's group holds bins 4 (l + 64 ic) .. + 3; the count in
        // higher lanes of the chunk is tot - inclusive prefix
        uint32_t my[4], mys = 0u;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if ((uint32_t)i == ic) {
#pragma unroll
                for (int e = 0; e < 4; ++e) my[e] = c[i][e];
                mys = cs[i];
            }
        const uint32_t inc = wave_incl_scan(mys);
        const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
        const uint32_t hi = above + tot - inc;           // count in bins above this lane's
        const uint64_t hit = __ballot(hi < kn && hi + mys >= kn);
        const int src = __builtin_ctzll(hit);
        uint32_t bs = 0u, run = hi;
#pragma unroll
        for (int e = 3; e >= 0; --e) {
            if (run < kn && run + my[e] >= kn) bs = 4u * ((uint32_t)lane + 64u * ic) + (uint32_t)e;
            run += my[e];
        }
        bloc = (uint32_t)__builtin_amdgcn_readlane((int)bs, src);
        if (lane == 0) s_bloc[wave] = bloc;
    }
    __syncthreads();

    // Local survivors in index order: WPH waves per head; wave k of head j holds
    // rows k * 64 * RPL .. of the region in RPL / 4 chunks of 256 rows, lane l
    // rows 4 l .. 4 l + 3 of each chunk (contiguous LDS reads), ranked chunk by
    // chunk with wave prefix sums.
    {
        constexpr int NC = RPL / 4;
        const int j = wave / WPH, k = wave - j * WPH;
        const int w0 = k * 64 * RPL;
        float sv[NC][4];
        uint32_t cnt[NC], pre[NC], wtot = 0u;
#pragma unroll
        for (int ch = 0; ch < NC; ++ch) {
            cnt[ch] = 0u;
            if (j < a.G) {
                const float4 x = *(const float4 *)&s_sc[j * kFilterRows + w0 + ch * 256 + 4 * lane];
                sv[ch][0] = x.x;
                sv[ch][1] = x.y;
                sv[ch][2] = x.z;
                sv[ch][3] = x.w;
                const uint32_t kmin = s_bloc[j] << kHistShift;
#pragma unroll
                for (int e = 0; e < 4; ++e) cnt[ch] += ord_key(sv[ch][e]) >= kmin ? 1u : 0u;
            }
            const uint32_t inc = wave_incl_scan(cnt[ch]);
            pre[ch] = wtot + inc - cnt[ch];
            wtot += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
        }
        if (lane == 0) s_wcnt[wave] = wtot;
        __syncthreads();
        if (j < a.G) {
            uint32_t off = 0u;
            for (int k2 = 0; k2 < k; ++k2) off += s_wcnt[j * WPH + k2];
            const uint32_t kmin = s_bloc[j] << kHistShift;
            uint64_t *dst = w.surv + (int64_t)(bh0 + j) * a.row_stride + r0;
#pragma unroll
            for (int ch = 0; ch < NC; ++ch) {
                uint32_t at = off + pre[ch];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (ord_key(sv[ch][e]) >= kmin)
                        dst[at++] = rank_of(sv[ch][e], (uint32_t)(r0 + w0 + ch * 256 + 4 * lane + e));
            }
            if (k == WPH - 1 && lane == 0) w.surv_cnt[(int64_t)(bh0 + j) * a.n_regions + f] = off + wtot;
        }
    }
    if (wave < a.G) {
        uint32_t *gh = w.hist + (int64_t)(bh0 + wave) * kHistBins;
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t bin = 4u * ((uint32_t)lane + 64u * (uint32_t)i) + (uint32_t)e;
                if (c[i][e] && bin >= bloc) atomicAdd(&gh[bin], c[i][e]);
            }
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

bool shape_supported(int dtype, int d, int g)
{
    return (dtype == 0 || dtype == 1) && (d == 64 || d == 128) && g >= 1 && g <= 8;
}

template <typename T, int D>
static void sim_desc(const StepArgs &a, KernelDesc *k)
{
    const int nsb = (a.M + kSimSlots - 1) / kSimSlots;
    // whole groups of 8 heads (one per XCD), nsb blocks each
    *k = KernelDesc{(const void *)&k_sim<T, D>, dim3((unsigned)((a.B * a.Hq + 7) / 8 * 8 * nsb)),
                    dim3(kSimThreads), 0u, 2};
}

template <typename T, int D, int G>
static void score_desc(const StepArgs &a, const Geometry &geo, KernelDesc *k)
{
    if constexpr (G <= 4) {
        if (geo.list_mode) {
            const unsigned blocks = (unsigned)((int64_t)a.B * a.Hkv * (a.len / kFilterRows));
            *k = KernelDesc{(const void *)&k_scan_list<T, D, G>, dim3(blocks),
                            dim3((unsigned)kListThreads<T, D, G>), (unsigned)scan_list_lds(G), 2};
            return;
        }
    }
    const unsigned blocks = (unsigned)(geo.scan_blocks + geo.cand_blocks);
    if (a.mode == MODE_SELECT) {
        const int n_merge = ((a.M + kSimSlots - 1) / kSimSlots) * a.R;
        const int r = score_range_lds(n_merge), c = score_scan_lds(G);
        *k = KernelDesc{(const void *)&k_score<T, D, G, true>, dim3(blocks), dim3(kScoreThreads),
                        (unsigned)(r > c ? r : c), 3};
    } else {
        *k = KernelDesc{(const void *)&k_score<T, D, G, false>, dim3(blocks), dim3(kScoreThreads),
                        (unsigned)score_scan_lds(G), 3};
    }
}

// k_final's geometry for a decode launch: slices per head so that the launch has
// about 256 blocks (one per CU; each block takes most of a CU's LDS), and 16
// entries per thread where a head's candidate cap is well past 4096 entries.
int final_slices(const StepArgs &a)
{
    const int bh = a.B * a.Hq;
    return bh <= 32 ? 8 : (bh <= 64 ? 4 : 2);
}
int final_ept(const StepArgs &a) { return (int64_t)a.R * a.K + a.W > 4608 ? 16 : 8; }

template <typename T, int D>
static void final_desc(const StepArgs &a, KernelDesc *k)
{
    if (a.U > 1) {
        *k = KernelDesc{(const void *)&k_final<T, D, true, 8, 8>, dim3((unsigned)(a.B * a.Hq * a.U)),
                        dim3(kFinalThreads), 0u, 2};
        return;
    }
    const int ns = final_slices(a), ept = final_ept(a);
    const void *f;
    if (ns == 8) f = ept == 8 ? (const void *)&k_final<T, D, false, 8, 8> : (const void *)&k_final<T, D, false, 8, 16>;
    else if (ns == 4) f = ept == 8 ? (const void *)&k_final<T, D, false, 4, 8> : (const void *)&k_final<T, D, false, 4, 16>;
    else f = ept == 8 ? (const void *)&k_final<T, D, false, 2, 8> : (const void *)&k_final<T, D, false, 2, 16>;
    // whole groups of 8 heads (one per XCD), ns blocks each
    *k = KernelDesc{f, dim3((unsigned)((a.B * a.Hq + 7) / 8 * 8 * ns)), dim3(kFinalThreads), 0u, 2};
}

// Group sizes run on the build for the next power of two (1, 2, 4 or 8); the
// extra heads pad the group.
template <typename T, int D>
static void score_g(const StepArgs &a, const Geometry &geo, KernelDesc *k)
{
    switch (a.G) {
    case 1: return score_desc<T, D, 1>(a, geo, k);
    case 2: return score_desc<T, D, 2>(a, geo, k);
    case 3: case 4: return score_desc<T, D, 4>(a, geo, k);
    default: return score_desc<T, D, 8>(a, geo, k);
    }
}

template <typename T, int D>
static void dense_g(const StepArgs &a, KernelDesc *k)
{
    const unsigned blocks = (unsigned)((int64_t)a.B * a.Hkv * ((a.len + kDenseRows - 1) / kDenseRows));
    const void *f;
    switch (a.G) {
    case 1: f = (const void *)&k_dense<T, D, 1>; break;
    case 2: f = (const void *)&k_dense<T, D, 2>; break;
    case 3: case 4: f = (const void *)&k_dense<T, D, 4>; break;
    default: f = (const void *)&k_dense<T, D, 8>; break;
    }
    *k = KernelDesc{f, dim3(blocks), dim3(kDenseThreads), 0u, 2};
}

void describe_kernel(int which, int dtype, const StepArgs &a, const Geometry &geo, KernelDesc *k)
{
    const bool bf = dtype == 1, d64 = a.D == 64;
    switch (which) {
    case KERNEL_SIM:
        if (bf) return d64 ? sim_desc<uint16_t, 64>(a, k) : sim_desc<uint16_t, 128>(a, k);
        return d64 ? sim_desc<float, 64>(a, k) : sim_desc<float, 128>(a, k);
    case KERNEL_SCORE:
        if (bf) return d64 ? score_g<uint16_t, 64>(a, geo, k) : score_g<uint16_t, 128>(a, geo, k);
        return d64 ? score_g<float, 64>(a, geo, k) : score_g<float, 128>(a, geo, k);
    case KERNEL_FILTER:
        // whole groups of 8 (virtual) heads, one per XCD
        *k = KernelDesc{(const void *)&k_filter,
                        dim3((unsigned)((a.B * a.Hq * a.U + 7) / 8 * 8 * geo.filter_blocks_per_head)),
                        dim3(kScoreThreads), 0u, 3};
        return;
    case KERNEL_PF_SCORE:   // bf16 only
        *k = KernelDesc{d64 ? (const void *)&k_pf_score<64> : (const void *)&k_pf_score<128>,
                        dim3((unsigned)(((geo.pf_pairs + 7) / 8) * 8 * geo.pf_qtiles)),
                        dim3(kPfThreads), 0u, 3};
        return;
    case KERNEL_DENSE:
        if (bf) return d64 ? dense_g<uint16_t, 64>(a, k) : dense_g<uint16_t, 128>(a, k);
        return d64 ? dense_g<float, 64>(a, k) : dense_g<float, 128>(a, k);
    case KERNEL_DENSE_MERGE:
        *k = KernelDesc{d64 ? (const void *)&k_dense_merge<64> : (const void *)&k_dense_merge<128>,
                        dim3((unsigned)(a.B * a.Hq)), dim3(kMergeThreads), 0u, 2};
        return;
    default:
        if (bf) return d64 ? final_desc<uint16_t, 64>(a, k) : final_desc<uint16_t, 128>(a, k);
        return d64 ? final_desc<float, 64>(a, k) : final_desc<float, 128>(a, k);
    }
}

}  // namespace retopk
