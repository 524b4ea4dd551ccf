// retopk_stream.hip -- a measurement aid, no part of the method: a plain
// streaming read of device memory, the practical HBM read ceiling that the
// benchmark reports beside the published peak (retopk_stream_read).
#include "retopk_internal.h"

namespace retopk {

// Every 16 bytes read once, eight loads per lane in flight, folded into one
// word per lane; the fold is stored only if it equals a value no real buffer of
// this size is expected to give, so that the loads are kept.
__global__ __launch_bounds__(512) void k_stream_read(const uint4 *p, int64_t n16, uint32_t *sink)
{
    constexpr int U = 8;
    const int64_t stride = (int64_t)gridDim.x * 512 * U;
    uint32_t acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * 512 * U + threadIdx.x; i < n16; i += stride) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t j = i + (int64_t)u * 512;
            v[u] = p[j < n16 ? j : 0];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;
}

void launch_stream_read(const void *src, int64_t bytes, uint32_t *sink, hipStream_t s)
{
    hipLaunchKernelGGL(k_stream_read, dim3(2048), dim3(512), 0, s, (const uint4 *)src, bytes / 16,
                       sink);
}

}  // namespace retopk
