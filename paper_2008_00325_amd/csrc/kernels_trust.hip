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
//  4. k_tw_rank: the input distances of blocks of 128 points to tiles of
//     columns as fp32 MFMA tiles (v_mfma_f32_16x16x4f32), turned into
//     distances in registers and compared with each point's neighbour
//     thresholds: only the counts r(i, j) - 1 leave the chip, never the n x n
//     distances.
//  5. k_tw_penalty: per-point penalty sum; k_tw_sum: one fixed-order reduction.
#include "internal.hpp"

namespace ul {

typedef float v4f __attribute__((ext_vector_type(4)));


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

// (distance, index) as one 64-bit key that orders as pair_less does for
// non-negative indices: the float's bits mapped to an unsigned integer of the
// same order (negative values flipped whole, positive ones with the sign bit
// set), -0 first made +0 so that equal floats give equal keys.
__device__ __forceinline__ uint64_t pair_key(float a, int32_t ia)
{
    const uint32_t bits = __float_as_uint(a + 0.0f);
    const uint32_t ord = (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
    return ((uint64_t)ord << 32) | (uint32_t)ia;
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

// One wavefront per point i: the input distance to each of its k embedding
// neighbours (lanes split the features, coalesced rows).  A neighbour slot
// left unfilled (a non-finite embedding coordinate never compares below the
// running threshold) raises `flags` and gets a threshold that nothing counts
// against.
__global__ __launch_bounds__(256) void k_tw_thresholds(const float *__restrict__ X, int64_t n, int32_t d, int32_t k,
                                                       const float *__restrict__ nx, const int32_t *__restrict__ nbr,
                                                       float *__restrict__ thr, unsigned *__restrict__ flags)
{
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) / kWave;
    const int lane = threadIdx.x % kWave;
    if (i >= n) return;   // whole waves
    const float *xi = X + i * d;
    for (int32_t s = 0; s < k; ++s) {
        const int64_t j = nbr[i * k + s];   // the same for every lane
        if (j < 0 || j >= n) {
            if (lane == 0) {
                thr[i * k + s] = -INFINITY;
                atomicOr(flags, 1u);
            }
            continue;
        }
        const float *xj = X + j * d;
        float dot = 0.0f;
        for (int32_t q = lane; q < d; q += kWave) dot = fmaf(xi[q], xj[q], dot);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) dot += __shfl_xor(dot, off);
        if (lane == 0) thr[i * k + s] = nx[i] + nx[j] - 2.0f * dot;
    }
}

// Input distances of a block of kRkRows points (rows) to a range of column
// tiles of CT x 16 points, as fp32 MFMA tiles (v_mfma_f32_16x16x4f32), turned
// into distances in registers and compared with each row's k thresholds.
//
//  * 8 waves; wave w owns rows 16 w .. 16 w + 15 of the block: lane l holds
//    row l % 16 and, in each of the CT column tiles of 16, the four columns
//    4 (l / 16) + 0..3 of the MFMA result layout.
//  * The features are taken CH (16 or 32) at a time, double buffered in LDS
//    ([point][feature], padded to CH + 4 floats so that a lane's 16-byte reads
//    are free of bank conflicts), the next chunk's global loads in flight while
//    the current one is multiplied.  Lane group g = l / 16 supplies features
//    g CH/4 .. (g + 1) CH/4 - 1, one per MFMA step, so each operand of a lane
//    comes from CH/16 16-byte LDS reads.
//  * Column splits (blockIdx.y) keep enough blocks in flight; each block adds
//    its rows' partial counts to cnt[row * k + s] with integer atomics (exact,
//    order-free).
constexpr int kRkRows = 128;
constexpr int kRankChunk = 16;   // features per LDS stage

__device__ __forceinline__ float4 load_features(const float *__restrict__ X, int64_t p, int32_t q, int64_t n,
                                                int32_t d, bool vec)
{
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (p >= n) return v;
    const float *x = X + p * d + q;
    if (vec) {
        if (q < d) v = *reinterpret_cast<const float4 *>(x);
    } else {
        if (q < d) v.x = x[0];
        if (q + 1 < d) v.y = x[1];
        if (q + 2 < d) v.z = x[2];
        if (q + 3 < d) v.w = x[3];
    }
    return v;
}

template <int KMAX, int CT, int CH>
__device__ __forceinline__ void rank_body(const float *__restrict__ X, int64_t n, int32_t d, int32_t k,
                                          const float *__restrict__ nx, const int32_t *__restrict__ nbr,
                                          const float *__restrict__ thr, int64_t tiles_per_split,
                                          int32_t *__restrict__ cnt_out)
{
    constexpr int COLS = 16 * CT;
    constexpr int PAD = CH + 4;        // floats per staged point
    constexpr int QUADS = CH / 4;      // float4 per staged point
    constexpr int NV = QUADS / 4;      // float4 a thread stages per operand (512 threads, 128 points)
    constexpr int GQ = CH / 16;        // float4 per lane group per operand
    static_assert(CH == 16 || CH == 32, "chunk of 16 or 32 features");
    __shared__ __align__(16) float s_rows[2][kRkRows * PAD];
    __shared__ __align__(16) float s_cols[2][COLS * PAD];
    __shared__ float s_nx[COLS];

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wv = tid / kWave;
    const int g = lane / 16;
    const int li = lane % 16;
    const int64_t row0 = (int64_t)blockIdx.x * kRkRows;
    const int rloc = wv * 16 + li;
    const int64_t row = row0 + rloc;
    const bool row_ok = row < n;
    const bool vec = (d % 4) == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0;   // 16-byte loads

    // each threshold as a (distance, index) key; an unused slot gets the
    // smallest key, which no element is below
    uint64_t tkey[KMAX];
    int32_t cnt[KMAX];
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
        const bool use = row_ok && s < k;
        tkey[s] = use ? pair_key(thr[row * k + s], nbr[row * k + s]) : 0ull;
        cnt[s] = 0;
    }
    const float nrow = row_ok ? nx[row] : 0.0f;

    // staging: float4 number f = tid + 512 v (v < NV) is features
    // 4 (f % QUADS) .. +3 of point f / QUADS
    int sp[NV], sq[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        sp[v] = (tid + 512 * v) / QUADS;
        sq[v] = 4 * ((tid + 512 * v) % QUADS);
    }
    const int64_t n_tiles = (n + COLS - 1) / COLS;
    const int64_t t0 = (int64_t)blockIdx.y * tiles_per_split;
    const int64_t t1 = t0 + tiles_per_split < n_tiles ? t0 + tiles_per_split : n_tiles;

    for (int64_t tile = t0; tile < t1; ++tile) {
        const int64_t col0 = tile * COLS;
        if (tid < COLS) s_nx[tid] = col0 + tid < n ? nx[col0 + tid] : 0.0f;
        v4f acc[CT];
#pragma unroll
        for (int t = 0; t < CT; ++t) acc[t] = v4f{0.0f, 0.0f, 0.0f, 0.0f};

        float4 rv[NV], cv[NV];
        auto fetch = [&](int32_t q0) __attribute__((always_inline)) {
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                rv[v] = load_features(X, row0 + sp[v], q0 + sq[v], n, d, vec);
                cv[v] = sp[v] < COLS ? load_features(X, col0 + sp[v], q0 + sq[v], n, d, vec)
                                     : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
        };
        auto stash = [&](int b) __attribute__((always_inline)) {
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                *reinterpret_cast<float4 *>(&s_rows[b][sp[v] * PAD + sq[v]]) = rv[v];
                if (sp[v] < COLS) *reinterpret_cast<float4 *>(&s_cols[b][sp[v] * PAD + sq[v]]) = cv[v];
            }
        };
        fetch(0);
        stash(0);
        __syncthreads();
        int buf = 0;
        for (int32_t q0 = 0; q0 < d; q0 += CH) {
            const bool more = q0 + CH < d;
            if (more) fetch(q0 + CH);
#pragma unroll
            for (int gq = 0; gq < GQ; ++gq) {
                const int f = g * (CH / 4) + 4 * gq;   // this lane group's features f .. f + 3
                const float4 bq = *reinterpret_cast<const float4 *>(&s_rows[buf][rloc * PAD + f]);
                float4 aq[CT];
#pragma unroll
                for (int t = 0; t < CT; ++t)
                    aq[t] = *reinterpret_cast<const float4 *>(&s_cols[buf][(t * 16 + li) * PAD + f]);
#pragma unroll
                for (int t = 0; t < CT; ++t) {
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq[t].x, bq.x, acc[t], 0, 0, 0);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq[t].y, bq.y, acc[t], 0, 0, 0);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq[t].z, bq.z, acc[t], 0, 0, 0);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq[t].w, bq.w, acc[t], 0, 0, 0);
                }
            }
            if (more) stash(buf ^ 1);
            __syncthreads();
            buf ^= 1;
        }
        if (row_ok) {
#pragma unroll
            for (int t = 0; t < CT; ++t) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int cl = t * 16 + 4 * g + e;
                    const int64_t c = col0 + cl;
                    if (c >= n || c == row) continue;
                    const float dist = nrow + s_nx[cl] - 2.0f * acc[t][e];
                    const int32_t ci = (int32_t)c;
                    const uint64_t key = pair_key(dist, ci);
                    // points ordered before neighbour s, the neighbour itself excluded (its
                    // distance here need not equal the threshold's bit for bit)
#pragma unroll
                    for (int s = 0; s < KMAX; ++s)
                        cnt[s] += (key < tkey[s] && (uint32_t)ci != (uint32_t)tkey[s]) ? 1 : 0;
                }
            }
        }
        __syncthreads();   // s_nx and the buffers are refilled for the next tile
    }
    // the four lanes of a row (l, l + 16, l + 32, l + 48) hold disjoint columns
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
        int32_t c = cnt[s];
        c += __shfl_xor(c, 16);
        c += __shfl_xor(c, 32);
        if (row_ok && g == 0 && s < k && c != 0) atomicAdd(&cnt_out[row * k + s], c);
    }
}

// pen[i] = sum_s max(0, r(i, nbr_s) - k), r = 1 + the count of points before
// the neighbour.
__global__ __launch_bounds__(256) void k_tw_penalty(const int32_t *__restrict__ cnt, int64_t n, int32_t k,
                                                    int64_t *__restrict__ pen)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    int64_t p = 0;
    for (int32_t s = 0; s < k; ++s) {
        const int64_t rank = (int64_t)cnt[i * k + s] + 1;
        if (rank > k) p += rank - k;
    }
    pen[i] = p;
}

__global__ __launch_bounds__(256) void k_tw_zero(int32_t *__restrict__ p, int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < count; t += stride) p[t] = 0;
}

template <int KMAX, int CT, int CH>
__global__ __launch_bounds__(512) void k_tw_rank(const float *__restrict__ X, int64_t n, int32_t d, int32_t k,
                                                 const float *__restrict__ nx, const int32_t *__restrict__ nbr,
                                                 const float *__restrict__ thr, int64_t tiles_per_split,
                                                 int32_t *__restrict__ cnt_out)
{
    rank_body<KMAX, CT, CH>(X, n, d, k, nx, nbr, thr, tiles_per_split, cnt_out);
}

// The same for k <= 16, held to 128 registers: two blocks per CU, which this
// instance reaches without spilling (the wider ones would spill).
template <int KMAX, int CT, int CH>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_tw_rank_occ(
    const float *__restrict__ X, int64_t n, int32_t d, int32_t k, const float *__restrict__ nx,
    const int32_t *__restrict__ nbr, const float *__restrict__ thr, int64_t tiles_per_split,
    int32_t *__restrict__ cnt_out)
{
    rank_body<KMAX, CT, CH>(X, n, d, k, nx, nbr, thr, tiles_per_split, cnt_out);
}

template <int KMAX, int CT, int CH = kRankChunk>
static void launch_rank(const float *X, int64_t n, int32_t d, int32_t k, const float *nx, const int32_t *nbr,
                        const float *thr, int32_t *cnt, hipStream_t s)
{
    const int64_t row_blocks = (n + kRkRows - 1) / kRkRows;
    const int64_t n_tiles = (n + 16 * CT - 1) / (16 * CT);
    // at least ~2048 blocks when the columns allow it
    int64_t splits = (2048 + row_blocks - 1) / row_blocks;
    if (splits > n_tiles) splits = n_tiles;
    if (splits < 1) splits = 1;
    const int64_t per_split = (n_tiles + splits - 1) / splits;
    splits = (n_tiles + per_split - 1) / per_split;
    if constexpr (KMAX <= 16)
        hipLaunchKernelGGL((k_tw_rank_occ<KMAX, CT, CH>), dim3((unsigned)row_blocks, (unsigned)splits), dim3(512), 0,
                           s, X, n, d, k, nx, nbr, thr, per_split, cnt);
    else
        hipLaunchKernelGGL((k_tw_rank<KMAX, CT, CH>), dim3((unsigned)row_blocks, (unsigned)splits), dim3(512), 0, s,
                           X, n, d, k, nx, nbr, thr, per_split, cnt);
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
                                  float *nx, int32_t *nbr, float *thr, int32_t *cnt, int64_t *pen,
                                  unsigned long long *sum, unsigned *flags, hipStream_t s)
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
    hipLaunchKernelGGL(k_tw_thresholds, dim3((unsigned)((n * kWave + 255) / 256)), dim3(256), 0, s, X, n, d, k, nx,
                       nbr, thr, flags);
    const int64_t nk = n * k;
    hipLaunchKernelGGL(k_tw_zero, dim3((unsigned)((nk + 255) / 256 < 4096 ? (nk + 255) / 256 : 4096)), dim3(256), 0,
                       s, cnt, nk);
    if (k <= 16)
        launch_rank<16, 4>(X, n, d, k, nx, nbr, thr, cnt, s);
    else if (k <= 32)
        launch_rank<32, 4>(X, n, d, k, nx, nbr, thr, cnt, s);
    else
        launch_rank<64, 2>(X, n, d, k, nx, nbr, thr, cnt, s);
    hipLaunchKernelGGL(k_tw_penalty, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, cnt, n, k, pen);
    hipLaunchKernelGGL(k_tw_sum, dim3(1), dim3(256), 0, s, pen, n, sum);
    return hipGetLastError();
}

}  // namespace ul
