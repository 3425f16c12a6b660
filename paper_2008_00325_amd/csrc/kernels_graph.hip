// kernels_graph.hip -- the input side of the layout: from kNN lists to the
// fuzzy union B (neighbourhood-weighting section, Eq. 1 and Eq. 2), in fp64.
//
//   k_dist_partial / k_dist_total  global mean distance (fixed-order sums,
//                                  used only to floor sigma of rows whose
//                                  distances are all zero)
//   k_smooth                       one thread per vertex: rho_i, then sigma_i
//                                  by bisection on sum_j exp(-(d_ij - rho_i)+ /
//                                  sigma) = log2 k, kept in registers (the
//                                  fused min / mean / search of the paper)
//   k_union                        one thread per kNN entry (i, s): A_ij, the
//                                  transposed value A_ji found by scanning
//                                  row j, and B_ij = A_ij + A_ji - A_ij A_ji
#include "internal.hpp"

namespace ul {

constexpr int kGraphTile = 4096;   // distances per partial sum

int64_t graph_partials(int64_t n, int32_t k) { return (n * k + kGraphTile - 1) / kGraphTile; }

__global__ __launch_bounds__(256) void k_dist_partial(const float *__restrict__ d, int64_t total,
                                                      double *__restrict__ partial)
{
    const int64_t base = (int64_t)blockIdx.x * kGraphTile;
    double s = 0.0;
    for (int t = threadIdx.x; t < kGraphTile; t += 256) {
        int64_t g = base + t;
        if (g < total) s += (double)d[g];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    __shared__ double s_w[4];
    if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) partial[blockIdx.x] = ((s_w[0] + s_w[1]) + s_w[2]) + s_w[3];
}

// One block: thread t adds partials t, t + 256, ... in order, then a fixed
// butterfly and a fixed sum over the four waves (the same order every call).
__global__ __launch_bounds__(256) void k_dist_total(double *partial, int64_t np)
{
    double s = 0.0;
    for (int64_t b = threadIdx.x; b < np; b += 256) s += partial[b];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    __shared__ double s_w[4];
    if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) partial[np] = ((s_w[0] + s_w[1]) + s_w[2]) + s_w[3];
}

__device__ __forceinline__ double membership(double dist, double rho, double sigma)
{
    double x = dist - rho;
    return exp(-(x > 0.0 ? x : 0.0) / sigma);
}

__global__ __launch_bounds__(256) void k_smooth(const int32_t *__restrict__ ids, const float *__restrict__ d,
                                                int64_t n, int32_t k, const double *__restrict__ partial,
                                                int64_t np, double *__restrict__ rho, double *__restrict__ sigma,
                                                unsigned *flags)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float *di = d + i * k;
    const int32_t *ii = ids + i * k;
    unsigned bad = 0;
    double r = 0.0, sum = 0.0;
    bool found = false;
    for (int32_t j = 0; j < k; ++j) {
        double dj = (double)di[j];
        if (!isfinite(di[j])) bad |= kBadValue;
        if ((uint32_t)ii[j] >= (uint32_t)n) bad |= kBadIndex;
        sum += dj;
        if (dj > 0.0 && (!found || dj < r)) {
            r = dj;
            found = true;
        }
    }
    if (bad) atomicOr(flags, bad);
    const double target = log2((double)k);
    double lo = 0.0, hi = INFINITY, s = 1.0;
    for (int it = 0; it < 64; ++it) {
        double f = 0.0;
        for (int32_t j = 0; j < k; ++j) {
            double x = (double)di[j] - r;
            f += x > 0.0 ? exp(-x / s) : 1.0;
        }
        if (fabs(f - target) < 1e-5) break;
        if (f > target) hi = s; else lo = s;
        s = isinf(hi) ? 2.0 * s : 0.5 * (lo + hi);
    }
    const double floor_v = found ? 1e-3 * (sum / (double)k) : 1e-3 * (partial[np] / ((double)n * (double)k));
    rho[i] = r;
    sigma[i] = s < floor_v ? floor_v : s;
}

__global__ __launch_bounds__(256) void k_union(const int32_t *__restrict__ ids, const float *__restrict__ d, int64_t n,
                                               int32_t k, const double *__restrict__ rho,
                                               const double *__restrict__ sigma, int32_t *__restrict__ rows,
                                               int32_t *__restrict__ cols, float *__restrict__ vals)
{
    const int64_t nk = n * k;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= nk) return;
    const int32_t i = (int32_t)(t / k);
    const int32_t j = ids[t];
    float b = 0.0f;
    bool mutual = false;
    if ((uint32_t)j < (uint32_t)n && j != i) {
        const double aij = membership((double)d[t], rho[i], sigma[i]);
        double aji = 0.0;
        const int64_t jb = (int64_t)j * k;
        for (int32_t s2 = 0; s2 < k; ++s2)
            if (ids[jb + s2] == i) {
                aji = membership((double)d[jb + s2], rho[j], sigma[j]);
                mutual = true;
            }
        b = (float)(aij + aji - aij * aji);
    }
    rows[t] = i;
    cols[t] = j;
    vals[t] = b;
    // the reverse orientation, unless row j lists i itself
    rows[nk + t] = mutual ? i : j;
    cols[nk + t] = i;
    vals[nk + t] = mutual ? 0.0f : b;
}

hipError_t launch_fuzzy_graph(int64_t n, int32_t k, const int32_t *ids, const float *dists, int32_t *rows,
                              int32_t *cols, float *vals, double *rho, double *sigma, double *partial,
                              int64_t npartial, unsigned *flags, hipStream_t s)
{
    const int64_t nk = n * k;
    hipLaunchKernelGGL(k_dist_partial, dim3((unsigned)npartial), dim3(256), 0, s, dists, nk, partial);
    hipLaunchKernelGGL(k_dist_total, dim3(1), dim3(256), 0, s, partial, npartial);
    hipLaunchKernelGGL(k_smooth, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, ids, dists, n, k, partial,
                       npartial, rho, sigma, flags);
    hipLaunchKernelGGL(k_union, dim3((unsigned)((nk + 255) / 256)), dim3(256), 0, s, ids, dists, n, k, rho, sigma,
                       rows, cols, vals);
    return hipGetLastError();
}

}  // namespace ul
