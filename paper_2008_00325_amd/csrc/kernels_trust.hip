// kernels_trust.hip -- trustworthiness T(k) of an embedding on the GPU
// (batched pairwise distances, Alg. 1; normalised as in Venna and Kaski's
// definition that the experiments section cites):
//
//   T(k) = 1 - 2 / (n k (2n - 3k - 1)) * sum_i sum_{j in N^_k(i)} max(0, r(i, j) - k)
//
// where N^_k(i) are the k nearest neighbours of i in the embedding and r(i, j)
// is the 1-based rank of j among all points by input distance from i (self
// excluded, ties by index); neighbours with r <= k are the input neighbours
// and add nothing.
//
//  1. k_tw_norms: |x_i|^2 of every input row.
//  2. k_tw_embed_knn: one wavefront per point, a brute-force scan of the
//     embedding keeping the k best (distance, index) pairs sorted across lanes.
//  3. k_tw_thresholds: input distance from i to each embedding neighbour.
//  4. k_tw_rank: the input distances of a block of 64 points to all n points as
//     fp32 MFMA tiles (v_mfma_f32_16x16x4f32), turned into distances in
//     registers and compared with each point's neighbour thresholds: only the
//     counts r(i, j) - 1 leave the chip, never the n x n distances.
//  5. k_tw_penalty: per-point penalty sum, then one fixed-order reduction.
#include "internal.hpp"

namespace ul {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kTwRows = 64;    // points per rank block (4 waves x 16)
constexpr int kTwCols = 64;    // column tile (4 MFMA tiles of 16)
constexpr int kTwChunk = 16;   // input features per LDS chunk (4 MFMA k-steps)

__global__ __launch_bounds__(256) void k_tw_norms(const float *__restrict__ X, int64_t n, int32_t d,
                                                  float *__restrict__ nx)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float *x = X + i * d;
    float s = 0.0f;
    for (int32_t q = 0; q < d; ++q) s = fmaf(x[q], x[q], s);
    nx[i] = s;
}

// (a, ia) before (b, ib): smaller distance, then smaller index.
__device__ __forceinline__ bool pair_less(float a, int32_t ia, float b, int32_t ib)
{
    return a < b || (a == b && ia < ib);
}

// One wavefront per point i: lanes 0..k-1 hold the k best (distance, index)
// pairs seen so far, ascending; each chunk of 64 candidates is merged by
// inserting the qualifying lanes one at a time.
template <int DIM>
__global__ __launch_bounds__(256) void k_tw_embed_knn(const float *__restrict__ Y, int64_t n, int32_t k,
                                                      int32_t *__restrict__ nbr)
{
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) / kWave;
    if (i >= n) return;
    const int lane = (int)(threadIdx.x % kWave);
    float yi[DIM];
#pragma unroll
    for (int q = 0; q < DIM; ++q) yi[q] = Y[i * DIM + q];
    float bd = INFINITY;
    int32_t bi = 0x7FFFFFFF;
    for (int64_t base = 0; base < n; base += kWave) {
        const int64_t c = base + lane;
        float dc = INFINITY;
        if (c < n && c != i) {
            dc = 0.0f;
#pragma unroll
            for (int q = 0; q < DIM; ++q) {
                const float t = Y[c * DIM + q] - yi[q];
                dc = fmaf(t, t, dc);
            }
        }
        const int32_t ci = (int32_t)c;
        bool pending = c < n && c != i;
        while (true) {
            const float td = __shfl(bd, k - 1);
            const int32_t ti = __shfl(bi, k - 1);
            pending = pending && pair_less(dc, ci, td, ti);
            const unsigned long long m = __ballot(pending);
            if (m == 0) break;
            const int src = __ffsll((long long)m) - 1;
            const float nd = __shfl(dc, src);
            const int32_t ni = __shfl(ci, src);
            if (lane == src) pending = false;
            // insertion position: slots holding a smaller pair
            const int pos = __popcll(__ballot(lane < k && pair_less(bd, bi, nd, ni)));
            const float up_d = __shfl_up(bd, 1);
            const int32_t up_i = __shfl_up(bi, 1);
            if (lane < k) {
                if (lane == pos) {
                    bd = nd;
                    bi = ni;
                } else if (lane > pos) {
                    bd = up_d;
                    bi = up_i;
                }
            }
        }
    }
    if (lane < k) nbr[i * k + lane] = bi;
}

// A neighbour slot left unfilled (a non-finite embedding coordinate never
// compares below the running threshold) raises `flags` and gets a threshold
// that nothing counts against.
__global__ __launch_bounds__(256) void k_tw_thresholds(const float *__restrict__ X, int64_t n, int32_t d, int32_t k,
                                                       const float *__restrict__ nx, const int32_t *__restrict__ nbr,
                                                       float *__restrict__ thr, unsigned *__restrict__ flags)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= n * k) return;
    const int64_t i = t / k;
    const int64_t j = nbr[t];
    if (j < 0 || j >= n) {
        thr[t] = -INFINITY;
        atomicOr(flags, 1u);
        return;
    }
    const float *xi = X + i * d;
    const float *xj = X + j * d;
    float dot = 0.0f;
    for (int32_t q = 0; q < d; ++q) dot = fmaf(xi[q], xj[q], dot);
    thr[t] = nx[i] + nx[j] - 2.0f * dot;
}

// Block: 64 points (rows) x all n points (columns), 4 waves of 16 rows.
// Lane l of a wave owns row (wave base + l % 16) and, in each of the 4 column
// sub-tiles, the 4 columns 4 * (l / 16) + 0..3 of the MFMA result layout.
template <int KMAX>
__global__ __launch_bounds__(256) void k_tw_rank(const float *__restrict__ X, int64_t n, int32_t d, int32_t k,
                                                 const float *__restrict__ nx, const int32_t *__restrict__ nbr,
                                                 const float *__restrict__ thr, int64_t *__restrict__ pen)
{
    __shared__ float s_rows[kTwChunk][kTwRows];   // [feature][row]
    __shared__ float s_cols[kTwChunk][kTwCols];   // [feature][column]

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wv = tid / kWave;
    const int64_t row0 = (int64_t)blockIdx.x * kTwRows;
    const int rloc = wv * 16 + (lane & 15);
    const int64_t row = row0 + rloc;
    const bool row_ok = row < n;

    float th[KMAX];
    int32_t nb[KMAX];
    int32_t cnt[KMAX];
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
        const bool use = row_ok && s < k;
        th[s] = use ? thr[row * k + s] : -INFINITY;
        nb[s] = use ? nbr[row * k + s] : -1;
        cnt[s] = 0;
    }
    const float nrow = row_ok ? nx[row] : 0.0f;

    // staging: thread tid loads feature (tid % 16) of point (tid / 16) + 16 m
    const int lq = tid % kTwChunk;
    const int lp = tid / kTwChunk;   // 0..15
    for (int64_t col0 = 0; col0 < n; col0 += kTwCols) {
        v4f acc[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
        for (int32_t q0 = 0; q0 < d; q0 += kTwChunk) {
            const int32_t q = q0 + lq;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int p = lp + 16 * m;
                const int64_t r = row0 + p;
                const int64_t c = col0 + p;
                s_rows[lq][p] = (q < d && r < n) ? X[r * d + q] : 0.0f;
                s_cols[lq][p] = (q < d && c < n) ? X[c * d + q] : 0.0f;
            }
            __syncthreads();
#pragma unroll
            for (int ks = 0; ks < kTwChunk; ks += 4) {
                const float b = s_rows[ks + lane / 16][wv * 16 + (lane & 15)];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const float a = s_cols[ks + lane / 16][t * 16 + (lane & 15)];
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[t], 0, 0, 0);
                }
            }
            __syncthreads();
        }
        if (!row_ok) continue;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t c = col0 + t * 16 + 4 * (lane / 16) + e;
                if (c >= n || c == row) continue;
                const float dist = nrow + nx[c] - 2.0f * acc[t][e];
                const int32_t ci = (int32_t)c;
#pragma unroll
                for (int s = 0; s < KMAX; ++s)
                    cnt[s] += (ci != nb[s] && pair_less(dist, ci, th[s], nb[s])) ? 1 : 0;
            }
        }
    }
    // the four lanes of a row (l, l + 16, l + 32, l + 48) hold disjoint columns
    int64_t p = 0;
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
        int32_t c = cnt[s];
        c += __shfl_xor(c, 16);
        c += __shfl_xor(c, 32);
        const int64_t rank = (int64_t)c + 1;
        if (s < k && rank > k) p += rank - k;
    }
    if (row_ok && lane < 16) pen[row] = p;
}

// Sum of pen[0..n) in a fixed order: one block, strided partial sums, then a
// tree.
__global__ __launch_bounds__(256) void k_tw_sum(const int64_t *__restrict__ pen, int64_t n,
                                                unsigned long long *__restrict__ out)
{
    __shared__ unsigned long long s_part[256];
    unsigned long long s = 0;
    for (int64_t t = threadIdx.x; t < n; t += 256) s += (unsigned long long)pen[t];
    s_part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s_part[threadIdx.x] += s_part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = s_part[0];
}

template <int DIM>
static hipError_t launch_knn_dim(const float *Y, int64_t n, int32_t k, int32_t *nbr, hipStream_t s)
{
    const int64_t blocks = (n * kWave + 255) / 256;
    hipLaunchKernelGGL((k_tw_embed_knn<DIM>), dim3((unsigned)blocks), dim3(256), 0, s, Y, n, k, nbr);
    return hipGetLastError();
}

hipError_t launch_trustworthiness(const float *X, int64_t n, int32_t d, const float *Y, int32_t dim, int32_t k,
                                  float *nx, int32_t *nbr, float *thr, int64_t *pen, unsigned long long *sum,
                                  unsigned *flags, hipStream_t s)
{
    hipLaunchKernelGGL(k_tw_norms, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, X, n, d, nx);
    hipError_t e = hipSuccess;
    switch (dim) {
#define UL_CASE(D) \
    case D: e = launch_knn_dim<D>(Y, n, k, nbr, s); break;
        UL_CASE(1) UL_CASE(2) UL_CASE(3) UL_CASE(4) UL_CASE(5) UL_CASE(6) UL_CASE(7) UL_CASE(8)
        UL_CASE(9) UL_CASE(10) UL_CASE(11) UL_CASE(12) UL_CASE(13) UL_CASE(14) UL_CASE(15) UL_CASE(16)
#undef UL_CASE
    default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_tw_thresholds, dim3((unsigned)((n * k + 255) / 256)), dim3(256), 0, s, X, n, d, k, nx, nbr,
                       thr, flags);
    const unsigned blocks = (unsigned)((n + kTwRows - 1) / kTwRows);
    if (k <= 16)
        hipLaunchKernelGGL((k_tw_rank<16>), dim3(blocks), dim3(256), 0, s, X, n, d, k, nx, nbr, thr, pen);
    else if (k <= 32)
        hipLaunchKernelGGL((k_tw_rank<32>), dim3(blocks), dim3(256), 0, s, X, n, d, k, nx, nbr, thr, pen);
    else
        hipLaunchKernelGGL((k_tw_rank<64>), dim3(blocks), dim3(256), 0, s, X, n, d, k, nx, nbr, thr, pen);
    hipLaunchKernelGGL(k_tw_sum, dim3(1), dim3(256), 0, s, pen, n, sum);
    return hipGetLastError();
}

}  // namespace ul
