// kernels_layout.hip -- random initialisation and the epoch kernels of the
// layout SGD (UMAP section objective; embedding-updates section), gfx950.
//
// Both epoch kernels implement one epoch-synchronous step: every read sees the
// snapshot E_n, every vertex's updates are summed in a fixed-point int64
// accumulator, and E_{n+1} = E_n + alpha * sum is written to the other buffer
// (no scatter to global memory, no global atomics on the embedding).
//  * k_epoch_wave:    edge-parallel.  Each wavefront owns a range of whole rows
//                     (balanced by edges + rows).  It streams the rows' eps in
//                     64-edge chunks, compacts the sampled edges into an LDS
//                     queue, and runs full 64-lane batches in which each lane
//                     handles one sampled edge: its attraction and its
//                     negative samples.  Sums go to a per-wave LDS accumulator
//                     with 64-bit integer atomics; the wave then writes its
//                     rows of E_{n+1} with coalesced stores.
//  * k_epoch_rowwise: one thread per vertex walking its row (a plain second
//                     implementation used to cross-check the first).
#include "internal.hpp"

namespace ul {

// ---------------------------------------------------------------------------
// Initial layout: uniform on [-10, 10) from the init stream.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_init(float *__restrict__ E, int64_t total, int32_t dim, uint32_t key_lo,
                                              uint32_t key_hi)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        int64_t i = t / dim;
        int32_t d = (int32_t)(t - i * dim);
        Ctr c;
        c.w[0] = (uint32_t)(uint64_t)i;
        c.w[1] = (uint32_t)((uint64_t)i >> 32);
        c.w[2] = (uint32_t)(d >> 2);
        c.w[3] = kTagInit;
        Ctr w = philox4x32_10(c, key_lo, key_hi);
        int sel = d & 3;
        uint32_t u = sel == 0 ? w.w[0] : sel == 1 ? w.w[1] : sel == 2 ? w.w[2] : w.w[3];
        // top 24 bits -> exact value in [-1, 1), then one fp32 rounding
        float unit = (float)((int32_t)(u >> 8) - (1 << 23)) * 0x1p-23f;
        E[t] = unit * 10.0f;
    }
}

hipError_t launch_init(float *E, int64_t n, int32_t dim, uint64_t seed, hipStream_t s)
{
    int64_t total = n * dim;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_init, dim3((unsigned)blocks), dim3(256), 0, s, E, total, dim, (uint32_t)seed,
                       (uint32_t)(seed >> 32));
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// One thread per vertex.
// ---------------------------------------------------------------------------
template <int DIM>
__global__ __launch_bounds__(256) void k_epoch_rowwise(EpochArgs A, const int64_t *__restrict__ row_ptr,
                                                       const int32_t *__restrict__ col,
                                                       const float *__restrict__ eps)
{
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    unsigned long long cnt = 0;
    if (i < A.n) {
        float yi[DIM];
#pragma unroll
        for (int d = 0; d < DIM; ++d) yi[d] = A.E[(size_t)i * DIM + d];
        long long acc[DIM];
#pragma unroll
        for (int d = 0; d < DIM; ++d) acc[d] = 0;
        const int64_t e1 = row_ptr[i + 1];
        for (int64_t e = row_ptr[i]; e < e1; ++e) {
            if (!edge_active(eps[e], A.epoch)) continue;
            long long fx[DIM];
            edge_contribution<DIM>(A, e, i, (uint32_t)col[e], yi, fx);
#pragma unroll
            for (int d = 0; d < DIM; ++d) acc[d] += fx[d];
            ++cnt;
        }
#pragma unroll
        for (int d = 0; d < DIM; ++d) A.E_next[(size_t)i * DIM + d] = commit(yi[d], acc[d], A.alpha);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    if ((threadIdx.x & 63) == 0 && cnt) atomicAdd(A.active_count, cnt);
}

// ---------------------------------------------------------------------------
// Edge-parallel wavefront kernel.
// ---------------------------------------------------------------------------
constexpr int kWavesPerBlock = 4;

// One batch: lane l handles queued edge q (if `valid`).  The head row is
// found by binary search in the wave's LDS copy of row_ptr.
template <int DIM>
__device__ __forceinline__ void wave_batch(const EpochArgs &A, const int32_t *__restrict__ col,
                                           const int64_t *rp, int nrows, int64_t r0, int64_t e0,
                                           long long *acc, int32_t off, bool valid)
{
    if (!valid) return;
    const int64_t e = e0 + off;
    int lo = 0, hi = nrows - 1;   // largest h with rp[h] <= e
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (rp[mid] <= e) lo = mid; else hi = mid - 1;
    }
    const uint32_t i = (uint32_t)(r0 + lo);
    float yi[DIM];
#pragma unroll
    for (int d = 0; d < DIM; ++d) yi[d] = A.E[(size_t)i * DIM + d];
    long long fx[DIM];
    edge_contribution<DIM>(A, e, i, (uint32_t)col[e], yi, fx);
#pragma unroll
    for (int d = 0; d < DIM; ++d)
        atomicAdd(reinterpret_cast<unsigned long long *>(&acc[lo * DIM + d]), (unsigned long long)fx[d]);
}

template <int DIM>
__global__ __launch_bounds__(256) void k_epoch_wave(EpochArgs A, const int64_t *__restrict__ row_ptr,
                                                    const int32_t *__restrict__ col,
                                                    const float *__restrict__ eps,
                                                    const int32_t *__restrict__ part, int64_t n_waves)
{
    constexpr int CAP = rows_cap(DIM);
    __shared__ long long s_acc[kWavesPerBlock][CAP * DIM];
    __shared__ int64_t s_rp[kWavesPerBlock][CAP + 1];
    __shared__ int32_t s_q[kWavesPerBlock][2 * kWave];

    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous run of logical blocks so that neighbouring rows (and their
    // mostly-local neighbours) share one L2.
    const int64_t per_xcd = gridDim.x / 8;
    const int64_t lb = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    const int wv = threadIdx.x / kWave;
    const unsigned lane = threadIdx.x % kWave;
    const int64_t w = lb * kWavesPerBlock + wv;
    if (w >= n_waves) return;
    const int64_t r0 = part[w];
    const int nrows = (int)(part[w + 1] - r0);
    if (nrows <= 0) return;

    long long *acc = s_acc[wv];
    int64_t *rp = s_rp[wv];
    int32_t *q = s_q[wv];
    for (int t = lane; t <= nrows; t += kWave) rp[t] = row_ptr[r0 + t];
    for (int t = lane; t < nrows * DIM; t += kWave) acc[t] = 0;
    wave_sync();

    const int64_t e0 = rp[0], e1 = rp[nrows];
    int qn = 0;
    unsigned long long cnt = 0;
    for (int64_t base = e0; base < e1; base += kWave) {
        const int64_t e = base + lane;
        const bool act = e < e1 && edge_active(eps[e], A.epoch);
        const unsigned long long m = __ballot(act);
        if (act) q[qn + lanes_below(m)] = (int32_t)(e - e0);
        const int c = __popcll(m);
        qn += c;
        cnt += c;
        wave_sync();
        if (qn >= kWave) {
            wave_batch<DIM>(A, col, rp, nrows, r0, e0, acc, q[lane], true);
            wave_sync();
            if ((int)lane < qn - kWave) q[lane] = q[kWave + lane];
            qn -= kWave;
            wave_sync();
        }
    }
    if (qn > 0) wave_batch<DIM>(A, col, rp, nrows, r0, e0, acc, q[lane], (int)lane < qn);
    wave_sync();

    const size_t g0 = (size_t)r0 * DIM;
    for (int t = lane; t < nrows * DIM; t += kWave) A.E_next[g0 + t] = commit(A.E[g0 + t], acc[t], A.alpha);
    if (lane == 0 && cnt) atomicAdd(A.active_count, cnt);
}

template <int DIM>
static hipError_t launch_epoch_dim(int kernel, const EpochArgs &A, const int64_t *row_ptr, const int32_t *col,
                                   const float *eps, const int32_t *part, int64_t n_waves, hipStream_t s)
{
    if (kernel == 1) {
        int64_t blocks = ((int64_t)A.n + 255) / 256;
        hipLaunchKernelGGL(k_epoch_rowwise<DIM>, dim3((unsigned)blocks), dim3(256), 0, s, A, row_ptr, col, eps);
    } else {
        int64_t blocks = (n_waves + kWavesPerBlock - 1) / kWavesPerBlock;
        int64_t per_xcd = (blocks + 7) / 8;
        hipLaunchKernelGGL(k_epoch_wave<DIM>, dim3((unsigned)(per_xcd * 8)), dim3(256), 0, s, A, row_ptr, col, eps,
                           part, n_waves);
    }
    return hipGetLastError();
}

hipError_t launch_epoch(int kernel, int32_t dim, const EpochArgs &A, const int64_t *row_ptr, const int32_t *col,
                        const float *eps, const int32_t *part, int64_t n_waves, hipStream_t s)
{
    switch (dim) {
#define UL_CASE(D) \
    case D: return launch_epoch_dim<D>(kernel, A, row_ptr, col, eps, part, n_waves, s);
        UL_CASE(1) UL_CASE(2) UL_CASE(3) UL_CASE(4) UL_CASE(5) UL_CASE(6) UL_CASE(7) UL_CASE(8)
        UL_CASE(9) UL_CASE(10) UL_CASE(11) UL_CASE(12) UL_CASE(13) UL_CASE(14) UL_CASE(15) UL_CASE(16)
#undef UL_CASE
    default: return hipErrorInvalidValue;
    }
}

// ---------------------------------------------------------------------------
// Diagnostics: the schedule and the negative draws, by the same routines.
// ---------------------------------------------------------------------------
__global__ void k_debug_active(const float *__restrict__ eps, int64_t nnz, int32_t epoch, uint8_t *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nnz; e += stride)
        out[e] = edge_active(eps[e], epoch) ? 1 : 0;
}

hipError_t launch_debug_active(const float *eps, int64_t nnz, int32_t epoch, uint8_t *out, hipStream_t s)
{
    int64_t blocks = (nnz + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_debug_active, dim3((unsigned)blocks), dim3(256), 0, s, eps, nnz, epoch, out);
    return hipGetLastError();
}

__global__ void k_debug_negatives(uint32_t n, uint32_t key_lo, uint32_t key_hi, int32_t epoch, int64_t e_first,
                                  int64_t count, int32_t neg_rate, uint32_t *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < count; t += stride) {
        const int64_t e = e_first + t;
        for (int32_t q = 0; q * 4 < neg_rate; ++q) {
            Ctr w = negative_words(e, epoch, q, key_lo, key_hi);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (4 * q + tt >= neg_rate) break;
                out[t * neg_rate + 4 * q + tt] = word_to_vertex(w.w[tt], n);
            }
        }
    }
}

hipError_t launch_debug_negatives(uint32_t n, uint64_t seed, int32_t epoch, int64_t e_first, int64_t count,
                                  int32_t neg_rate, uint32_t *out, hipStream_t s)
{
    int64_t blocks = (count + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_debug_negatives, dim3((unsigned)blocks), dim3(256), 0, s, n, (uint32_t)seed,
                       (uint32_t)(seed >> 32), epoch, e_first, count, neg_rate, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Roofline probe: a plain 16-byte vector copy.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_probe_copy(const float4 *__restrict__ src, float4 *__restrict__ dst,
                                                    int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < count; t += stride) dst[t] = src[t];
}

hipError_t launch_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t s)
{
    int64_t count = bytes / 16;
    int64_t blocks = (count + 255) / 256;
    if (blocks > 256 * 64) blocks = 256 * 64;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_probe_copy, dim3((unsigned)blocks), dim3(256), 0, s, (const float4 *)src, (float4 *)dst,
                       count);
    return hipGetLastError();
}

}  // namespace ul
