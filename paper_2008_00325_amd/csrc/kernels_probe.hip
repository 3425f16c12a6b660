// kernels_probe.hip -- measurement probes for the roofline of the layout
// kernels: a plain 16-byte copy (the HBM ceiling, and the calibration of the
// FETCH_SIZE / WRITE_SIZE counters) and random 8-byte gathers from a table of
// a given size (the cache-served ceiling of the negative-sample gathers).
#include "internal.hpp"

namespace ul {

// ---------------------------------------------------------------------------
// Roofline probe: a plain 16-byte vector copy.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_probe_copy(const float4 *__restrict__ src, float4 *__restrict__ dst,
                                                    int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < count; t += stride) dst[t] = src[t];
}

// Random-gather probe: the same 8-byte gathers as the repulsions, positions
// from a 32-bit integer hash (lowbias32-style multiply-xorshift mixing) of
// (thread, step), masked to the table size.
__device__ __forceinline__ uint32_t mix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

__global__ __launch_bounds__(256) void k_probe_gather(const float2 *__restrict__ table, uint32_t mask, int32_t iters,
                                                      float *__restrict__ out)
{
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    uint32_t s = mix32(t * 0x9E3779B9u + 0x632BE5ABu);
    float acc = 0.0f;
    for (int32_t it = 0; it < iters; ++it) {
        float2 v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            s = s * 1664525u + 1013904223u;
            v[u] = table[mix32(s) & mask];
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += v[u].x * v[u].y;
    }
    if (acc == 1.0e30f) out[t] = acc;
}

hipError_t launch_probe_gather(const void *table, int64_t entries, int64_t threads, int32_t iters, void *out,
                               hipStream_t s)
{
    hipLaunchKernelGGL(k_probe_gather, dim3((unsigned)(threads / 256)), dim3(256), 0, s, (const float2 *)table,
                       (uint32_t)(entries - 1), iters, (float *)out);
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t s)
{
    // one 16-byte element per thread up to 2^18 blocks (1 GiB): with a
    // grid-stride loop over 64 blocks per CU the copy reached 4.6 TB/s, with
    // one element per thread 6.2 TB/s
    int64_t count = bytes / 16;
    int64_t blocks = (count + 255) / 256;
    if (blocks > 256 * 1024) blocks = 256 * 1024;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_probe_copy, dim3((unsigned)blocks), dim3(256), 0, s, (const float4 *)src, (float4 *)dst,
                       count);
    return hipGetLastError();
}

}  // namespace ul
