// kernels_prep.hip -- device ingest of the COO graph B (sparse-data handling
// section: the COO list is sorted by row and indexed by a CSR row pointer).
//
// Steps (all on the handle's stream, one host synchronisation at the end):
//   1. check indices and values; w_max = largest weight of a candidate edge
//      (val > 0, row != col; a bipartite graph -- new points to a frozen
//      table -- keeps row == col, which are different vertices there)
//   2. count kept edges per row (candidates with val >= w_max / n_epochs)
//   3. exclusive scan of the counts -> row_ptr (int64), largest row
//   4. scatter kept edges into their row's segment (order inside a row is
//      arbitrary at this point)
//   5. sort each row by column, and compute eps = w_max / val: rows of up to
//      kLongRow entries by a rank sort (the rank of an entry is the number of
//      smaller columns in its row; equal columns flag a duplicate), longer
//      rows by a stable radix sort of their columns, one workgroup per row
//      (equal neighbours after it flag a duplicate)
//   6. symmetry (not for a bipartite graph): each kept (i, j, v) must find
//      (j, i) with bit-equal v by binary search in row j
//   7. wave partition for the epoch kernel
#include "internal.hpp"

namespace ul {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

// rows in [0, n), columns in [0, n_cols); bipartite: row and column index
// different vertex sets
struct IngestShape {
    uint32_t n, n_cols;
    int32_t bipartite;
};

__device__ __forceinline__ bool candidate(int32_t r, int32_t c, float v, IngestShape sh)
{
    return (uint32_t)r < sh.n && (uint32_t)c < sh.n_cols && (sh.bipartite || r != c) && v > 0.0f && isfinite(v);
}

__device__ __forceinline__ float keep_threshold(const PrepScalars *S, int32_t n_epochs)
{
    return __uint_as_float(S->wmax_bits) / (float)n_epochs;
}

__device__ __forceinline__ unsigned wave_or(unsigned v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v |= __shfl_xor(v, off);
    return v;
}

__device__ __forceinline__ unsigned wave_max(unsigned v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = max(v, (unsigned)__shfl_xor(v, off));
    return v;
}

__global__ __launch_bounds__(256) void k_check_max(const int32_t *__restrict__ rows, const int32_t *__restrict__ cols,
                                                   const float *__restrict__ vals, int64_t nnz, IngestShape sh,
                                                   PrepScalars *S)
{
    unsigned flags = 0, mx = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nnz; t += stride) {
        int32_t r = rows[t], c = cols[t];
        float v = vals[t];
        if ((uint32_t)r >= sh.n || (uint32_t)c >= sh.n_cols) flags |= kBadIndex;
        if (!isfinite(v)) flags |= kBadValue;
        if (candidate(r, c, v, sh)) mx = max(mx, __float_as_uint(v));  // positive floats order as integers
    }
    // one atomic per block: every block has a candidate weight, and atomics
    // from thousands of waves on one address would serialise
    flags = wave_or(flags);
    mx = wave_max(mx);
    __shared__ unsigned s_flags[4], s_max[4];
    if ((threadIdx.x & 63) == 0) {
        s_flags[threadIdx.x >> 6] = flags;
        s_max[threadIdx.x >> 6] = mx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned f = s_flags[0] | s_flags[1] | s_flags[2] | s_flags[3];
        const unsigned m = max(max(s_max[0], s_max[1]), max(s_max[2], s_max[3]));
        if (f) atomicOr(&S->flags, f);
        if (m) atomicMax(&S->wmax_bits, m);
    }
}

// Slot of the calling lane in the counter ctr[key], with one atomic add per
// run of consecutive lanes that hold the same key (inactive lanes end a run):
// the counter's old value plus the lane's rank in its run.  Kernel-built
// graphs list a row's entries together, so runs are long.  Every lane of the
// wave must call it.
__device__ __forceinline__ int32_t run_atomic_add(int32_t *ctr, int32_t key, bool active)
{
    const int lane = (int)lane_id();
    const int32_t prev = __shfl_up(key, 1);
    const unsigned long long act = __ballot(active);
    const bool prev_act = lane > 0 && ((act >> (lane - 1)) & 1ull);
    const bool head = active && !(prev_act && prev == key);
    const unsigned long long heads = __ballot(head);
    const unsigned long long le = (2ull << lane) - 1ull;   // lanes 0 .. lane
    int32_t base = 0;
    if (head) {
        const unsigned long long above = (heads | ~act) & ~le;
        const int end = above ? __builtin_ctzll(above) : 64;
        base = atomicAdd(&ctr[key], end - lane);
    }
    const unsigned long long hm = heads & le;
    const int h = hm ? 63 - __builtin_clzll(hm) : lane;
    return __shfl(base, h) + lane - h;
}

__global__ __launch_bounds__(256) void k_count(const int32_t *__restrict__ rows, const int32_t *__restrict__ cols,
                                               const float *__restrict__ vals, int64_t nnz, IngestShape sh,
                                               int32_t n_epochs, const PrepScalars *S, int32_t *__restrict__ deg)
{
    const float thresh = keep_threshold(S, n_epochs);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    // wave-uniform trip count: run_atomic_add needs the whole wave
    for (int64_t t0 = (int64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~63u); t0 < nnz; t0 += stride) {
        const int64_t t = t0 + (threadIdx.x & 63u);
        const bool in = t < nnz;
        const int32_t r = in ? rows[t] : 0, c = in ? cols[t] : 0;
        const float v = in ? vals[t] : 0.0f;
        const bool keep = in && candidate(r, c, v, sh) && v >= thresh;
        run_atomic_add(deg, r, keep);
    }
}

// Inclusive scan of one value per thread across a 256-thread block.
__device__ __forceinline__ int64_t block_inclusive_scan(int64_t x, int64_t *s_wave)
{
    const unsigned lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int64_t y = __shfl_up(x, off);
        if (lane >= (unsigned)off) x += y;
    }
    if (lane == 63) s_wave[wv] = x;
    __syncthreads();
    int64_t add = 0;
    for (unsigned k = 0; k < wv; ++k) add += s_wave[k];
    __syncthreads();
    return x + add;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(const int32_t *__restrict__ deg, int64_t n,
                                                              int64_t *__restrict__ bsum, PrepScalars *S)
{
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int64_t s = 0;
    int mx = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k)
        if (base + k < n) {
            int v = deg[base + k];
            s += v;
            mx = max(mx, v);
        }
    __shared__ int64_t s_wave[4];
    int64_t inc = block_inclusive_scan(s, s_wave);
    if (threadIdx.x == kScanThreads - 1) bsum[blockIdx.x] = inc;
    mx = (int)wave_max((unsigned)mx);
    if ((threadIdx.x & 63) == 0 && mx) atomicMax(&S->max_degree, mx);
}

// Exclusive scan of the block sums in place (one block, loops over chunks).
__global__ __launch_bounds__(kScanThreads) void k_scan_top(int64_t *__restrict__ bsum, int64_t nb)
{
    __shared__ int64_t s_wave[4];
    __shared__ int64_t s_carry;
    if (threadIdx.x == 0) s_carry = 0;
    __syncthreads();
    for (int64_t base = 0; base < nb; base += kScanThreads) {
        int64_t t = base + threadIdx.x;
        int64_t v = t < nb ? bsum[t] : 0;
        int64_t inc = block_inclusive_scan(v, s_wave);
        int64_t carry = s_carry;
        if (t < nb) bsum[t] = carry + inc - v;
        __syncthreads();
        if (threadIdx.x == kScanThreads - 1) s_carry = carry + inc;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kScanThreads) void k_scan_down(const int32_t *__restrict__ deg, int64_t n,
                                                            const int64_t *__restrict__ boff,
                                                            int64_t *__restrict__ row_ptr, int64_t nb)
{
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = base + k < n ? deg[base + k] : 0;
        s += v[k];
    }
    __shared__ int64_t s_wave[4];
    int64_t run = block_inclusive_scan(s, s_wave) - s + boff[blockIdx.x];
#pragma unroll
    for (int k = 0; k < kScanItems; ++k)
        if (base + k < n) {
            row_ptr[base + k] = run;
            run += v[k];
        }
    // the last block also writes the total
    if (blockIdx.x == nb - 1 && threadIdx.x == kScanThreads - 1) row_ptr[n] = run;
}

__global__ __launch_bounds__(256) void k_scatter(const int32_t *__restrict__ rows, const int32_t *__restrict__ cols,
                                                 const float *__restrict__ vals, int64_t nnz, IngestShape sh,
                                                 int32_t n_epochs, const PrepScalars *S,
                                                 const int64_t *__restrict__ row_ptr, int32_t *__restrict__ cursor,
                                                 int32_t *__restrict__ trow, int32_t *__restrict__ tcol,
                                                 float *__restrict__ tval)
{
    const float thresh = keep_threshold(S, n_epochs);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t0 = (int64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~63u); t0 < nnz; t0 += stride) {
        const int64_t t = t0 + (threadIdx.x & 63u);
        const bool in = t < nnz;
        const int32_t r = in ? rows[t] : 0, c = in ? cols[t] : 0;
        const float v = in ? vals[t] : 0.0f;
        const bool keep = in && candidate(r, c, v, sh) && v >= thresh;
        const int32_t slot = run_atomic_add(cursor, r, keep);
        if (keep) {
            const int64_t p = row_ptr[r] + slot;
            trow[p] = r;
            tcol[p] = c;
            tval[p] = v;
        }
    }
}

// Rows longer than this are sorted by k_long_row_sort: the rank sort reads a
// row once per entry, deg^2 loads in all.
constexpr int64_t kLongRow = 2048;
constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / 64;

__global__ __launch_bounds__(256) void k_row_sort(const int32_t *__restrict__ trow, const int32_t *__restrict__ tcol,
                                                  const float *__restrict__ tval, const int64_t *__restrict__ row_ptr,
                                                  int64_t n, PrepScalars *S, int32_t *__restrict__ col,
                                                  float *__restrict__ sval, float *__restrict__ eps)
{
    const int64_t kept = row_ptr[n];
    const float w_max = __uint_as_float(S->wmax_bits);
    unsigned flags = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < kept; p += stride) {
        const int32_t r = trow[p];
        const int32_t c = tcol[p];
        const int64_t rs = row_ptr[r], re = row_ptr[r + 1];
        if (re - rs > kLongRow) continue;   // k_long_row_sort
        // rank of c in its row; eight loads of the row in flight at a time
        int64_t rank = 0;
        for (int64_t q0 = rs; q0 < re; q0 += 8) {
            int32_t cq[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) cq[u] = q0 + u < re ? tcol[q0 + u] : INT32_MAX;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                rank += cq[u] < c;
                if (cq[u] == c && q0 + u != p) flags |= kDuplicate;
            }
        }
        const int64_t dst = rs + rank;
        const float v = tval[p];
        col[dst] = c;
        sval[dst] = v;
        eps[dst] = w_max / v;
    }
    flags = wave_or(flags);
    if ((threadIdx.x & 63) == 0 && flags) atomicOr(&S->flags, flags);
}

// list[] = the rows longer than kLongRow, count[0] = how many (zeroed before).
__global__ __launch_bounds__(256) void k_long_rows(const int64_t *__restrict__ row_ptr, int64_t n,
                                                   int32_t *__restrict__ list, int32_t *count)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r < n && row_ptr[r + 1] - row_ptr[r] > kLongRow) list[atomicAdd(count, 1)] = (int32_t)r;
}

// One workgroup per long row: a least-significant-digit radix sort of the
// row's (column, slot) pairs by column, 4-bit digits, each pass stable (the
// digit's global offset from a counting sweep, then chunks of 1024 entries in
// order, each entry placed after the earlier entries of its digit: rank in
// its wavefront by ballot, wavefront offsets in LDS).  The pairs move between
// two buffers inside the row's own segment: (tcol, sval) and (col, eps) --
// sval and eps hold the slot as an int until the last step writes them.  An
// even number of passes leaves the result in (tcol, sval); then col, sval and
// eps are written in sorted order and equal neighbours flag a duplicate.
__global__ __launch_bounds__(kSortThreads) void k_long_row_sort(int32_t *__restrict__ tcol,
                                                                const float *__restrict__ tval,
                                                                const int64_t *__restrict__ row_ptr,
                                                                const int32_t *__restrict__ list,
                                                                const int32_t *__restrict__ count, int32_t passes,
                                                                PrepScalars *S, int32_t *__restrict__ col,
                                                                float *__restrict__ sval, float *__restrict__ eps)
{
    if ((int32_t)blockIdx.x >= *count) return;
    __shared__ int32_t s_hist[16];
    __shared__ int32_t s_wcnt[kSortWaves][16];
    __shared__ int32_t s_woff[kSortWaves][16];
    const int32_t r = list[blockIdx.x];
    const int64_t rs = row_ptr[r], L = row_ptr[r + 1] - rs;
    const int tid = threadIdx.x, wv = tid / 64, lane = tid % 64;
    int32_t *const key[2] = {tcol + rs, col + rs};
    int32_t *const idx[2] = {reinterpret_cast<int32_t *>(sval) + rs, reinterpret_cast<int32_t *>(eps) + rs};
    for (int64_t t = tid; t < L; t += kSortThreads) idx[0][t] = (int32_t)t;
    __syncthreads();
    for (int32_t pass = 0; pass < passes; ++pass) {
        const int src = pass & 1, dst = src ^ 1;
        const int shift = 4 * pass;
        if (tid < 16) s_hist[tid] = 0;
        __syncthreads();
        for (int64_t t = tid; t < L; t += kSortThreads) atomicAdd(&s_hist[((uint32_t)key[src][t] >> shift) & 15u], 1);
        __syncthreads();
        if (tid == 0) {
            int32_t run = 0;
            for (int d = 0; d < 16; ++d) {
                const int32_t c = s_hist[d];
                s_hist[d] = run;   // first slot of digit d
                run += c;
            }
        }
        __syncthreads();
        for (int64_t c0 = 0; c0 < L; c0 += kSortThreads) {
            const int64_t t = c0 + tid;
            const bool valid = t < L;
            const int32_t k = valid ? key[src][t] : 0;
            const int32_t ix = valid ? idx[src][t] : 0;
            const int d = valid ? (int)(((uint32_t)k >> shift) & 15u) : 16;
            int rank = 0;
            for (int v = 0; v < 16; ++v) {
                const unsigned long long m = __ballot(d == v);
                if (d == v) rank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                if (lane == 0) s_wcnt[wv][v] = __popcll(m);
            }
            __syncthreads();
            if (tid < 16) {
                int32_t run = s_hist[tid];
                for (int w = 0; w < kSortWaves; ++w) {
                    s_woff[w][tid] = run;
                    run += s_wcnt[w][tid];
                }
                s_hist[tid] = run;
            }
            __syncthreads();
            if (valid) {
                const int32_t pos = s_woff[wv][d] + rank;
                key[dst][pos] = k;
                idx[dst][pos] = ix;
            }
            __syncthreads();
        }
    }
    const float w_max = __uint_as_float(S->wmax_bits);
    unsigned flags = 0;
    for (int64_t t = tid; t < L; t += kSortThreads) {
        const int32_t c = key[0][t];
        const int32_t ix = idx[0][t];
        if (t > 0 && key[0][t - 1] == c) flags |= kDuplicate;
        const float v = tval[rs + ix];
        col[rs + t] = c;
        sval[rs + t] = v;
        eps[rs + t] = w_max / v;
    }
    flags = wave_or(flags);
    if (lane == 0 && flags) atomicOr(&S->flags, flags);
}

__global__ __launch_bounds__(256) void k_symmetry(const int32_t *__restrict__ trow, const int32_t *__restrict__ col,
                                                  const float *__restrict__ sval, const int64_t *__restrict__ row_ptr,
                                                  int64_t n, PrepScalars *S)
{
    // After a duplicate the in-row sort leaves some slots unwritten; the
    // graph is rejected anyway, so skip the check rather than read them.
    if (S->flags & (kDuplicate | kBadIndex | kBadValue)) return;
    const int64_t kept = row_ptr[n];
    unsigned flags = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < kept; p += stride) {
        const int32_t i = trow[p];   // row slots keep their row through the in-row sort
        const int32_t j = col[p];
        if ((uint32_t)j >= (uint32_t)n) {
            flags |= kAsymmetric;
            continue;
        }
        int64_t lo = row_ptr[j], hi = row_ptr[j + 1];
        const int64_t end = hi;
        while (lo < hi) {
            int64_t mid = (lo + hi) >> 1;
            if (col[mid] < i) lo = mid + 1; else hi = mid;
        }
        if (lo >= end || col[lo] != i || __float_as_uint(sval[lo]) != __float_as_uint(sval[p])) flags |= kAsymmetric;
    }
    flags = wave_or(flags);
    if ((threadIdx.x & 63) == 0 && flags) atomicOr(&S->flags, flags);
}

static int64_t grid_for(int64_t items)
{
    int64_t b = (items + 255) / 256;
    if (b > 256 * 32) b = 256 * 32;
    return b < 1 ? 1 : b;
}

int64_t scan_blocks(int64_t n) { return (n + kScanTile - 1) / kScanTile; }

hipError_t launch_prep(const PrepBuffers &B, hipStream_t s)
{
    const IngestShape sh{(uint32_t)B.n, (uint32_t)B.n_cols, B.bipartite ? 1 : 0};
    const int64_t g = grid_for(B.nnz);
    // a grid-stride pass with a block-wide reduction: 2048 blocks fill the chip
    const int64_t g_check = g < 2048 ? g : 2048;
    hipLaunchKernelGGL(k_check_max, dim3((unsigned)g_check), dim3(256), 0, s, B.rows, B.cols, B.vals, B.nnz, sh,
                       B.scalars);
    hipLaunchKernelGGL(k_count, dim3((unsigned)g), dim3(256), 0, s, B.rows, B.cols, B.vals, B.nnz, sh, B.n_epochs,
                       B.scalars, B.deg);
    const int64_t nb = B.nblocks_scan;
    hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, s, B.deg, B.n, B.bsum, B.scalars);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kScanThreads), 0, s, B.bsum, nb);
    hipLaunchKernelGGL(k_scan_down, dim3((unsigned)nb), dim3(kScanThreads), 0, s, B.deg, B.n, B.bsum, B.row_ptr, nb);
    hipLaunchKernelGGL(k_scatter, dim3((unsigned)g), dim3(256), 0, s, B.rows, B.cols, B.vals, B.nnz, sh, B.n_epochs,
                       B.scalars, B.row_ptr, B.cursor, B.trow, B.tcol, B.tval);
    hipLaunchKernelGGL(k_row_sort, dim3((unsigned)g), dim3(256), 0, s, B.trow, B.tcol, B.tval, B.row_ptr, B.n,
                       B.scalars, B.col, B.sval, B.eps);
    // rows longer than kLongRow: their list in deg (free after the scan), its
    // length in cursor[0] (free after the scatter)
    const int64_t max_long = B.nnz / (kLongRow + 1);
    if (max_long > 0) {
        int32_t passes = 0;   // 4-bit digits of the largest column, rounded up to an even count
        for (int64_t top = B.n_cols - 1; top > 0; top >>= 4) ++passes;
        passes += passes & 1;
        hipError_t e = hipMemsetAsync(B.cursor, 0, sizeof(int32_t), s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_long_rows, dim3((unsigned)((B.n + 255) / 256)), dim3(256), 0, s, B.row_ptr, B.n, B.deg,
                           B.cursor);
        const int64_t rows = max_long < B.n ? max_long : B.n;
        hipLaunchKernelGGL(k_long_row_sort, dim3((unsigned)rows), dim3(kSortThreads), 0, s, B.tcol, B.tval, B.row_ptr,
                           B.deg, B.cursor, passes, B.scalars, B.col, B.sval, B.eps);
    }
    if (!B.bipartite)
        hipLaunchKernelGGL(k_symmetry, dim3((unsigned)g), dim3(256), 0, s, B.trow, B.col, B.sval, B.row_ptr, B.n,
                           B.scalars);
    return hipGetLastError();
}

// part[w] = first row r with row_ptr[r] + wgt * r >= w * cost, for
// w < n_waves; part[n_waves] = n.  A wave then holds at most
// cost / wgt + 1 <= rows_cap(dim) rows (cost rises by >= wgt per row) and
// about cost edges unless its last row alone is longer.
// Waves over rows [r0, r1): part[w] is the first row r >= r0 whose units
// (edges and row weights from r0 up to r) reach w x cost; part[n_waves] = r1.
__global__ void k_partition(const int64_t *__restrict__ row_ptr, int64_t r0, int64_t r1, int32_t wgt, int64_t cost,
                            int32_t *__restrict__ part, int64_t n_waves)
{
    const int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (w > n_waves) return;
    if (w == n_waves) {
        part[w] = (int32_t)r1;
        return;
    }
    const int64_t target = row_ptr[r0] + (int64_t)wgt * r0 + w * cost;
    int64_t lo = r0, hi = r1;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (row_ptr[mid] + (int64_t)wgt * mid >= target) hi = mid; else lo = mid + 1;
    }
    part[w] = (int32_t)lo;
}

// head[e] = row of edge e minus the first row of its wave (< rows_cap <= 256).
// One thread per row of [r0, r1): its wave is the last w with part[w] <= row.
__global__ void k_head_local(const int64_t *__restrict__ row_ptr, int64_t r0, int64_t r1,
                             const int32_t *__restrict__ part, int64_t n_waves, uint8_t *__restrict__ head)
{
    const int64_t r = r0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= r1) return;
    int64_t lo = 0, hi = n_waves - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi + 1) >> 1;
        if (part[mid] <= r) lo = mid; else hi = mid - 1;
    }
    const uint8_t h = (uint8_t)(r - part[lo]);
    for (int64_t e = row_ptr[r]; e < row_ptr[r + 1]; ++e) head[e] = h;
}

hipError_t launch_partition(const int64_t *row_ptr, int64_t r0, int64_t r1, int32_t dim, int64_t cost,
                            int32_t *part, int64_t n_waves, uint8_t *head, hipStream_t s)
{
    if (cost < 1 || cost > kWaveCost || r0 < 0 || r1 <= r0 || n_waves < 1) return hipErrorInvalidValue;
    static_assert(rows_cap(1) <= 256 && rows_cap(16) <= 256, "head offsets must fit in a byte");
    int64_t blocks = (n_waves + 1 + 255) / 256;
    hipLaunchKernelGGL(k_partition, dim3((unsigned)blocks), dim3(256), 0, s, row_ptr, r0, r1, row_weight(dim), cost,
                       part, n_waves);
    hipLaunchKernelGGL(k_head_local, dim3((unsigned)((r1 - r0 + 255) / 256)), dim3(256), 0, s, row_ptr, r0, r1, part,
                       n_waves, head);
    return hipGetLastError();
}

// delta[e] = col[e] - (row of e) in 16 bits; *wide gets 1 when some delta
// does not fit (then the wave kernels read the 32-bit columns and delta is not
// used).  One block per 256 rows reads and writes the rows' edges with
// consecutive threads on consecutive edges and finds each edge's row by a
// binary search over the rows' starts staged in LDS (one thread walking a
// whole row waits on one load per edge: 454 us at 1M vertices, k = 15).
__global__ __launch_bounds__(256) void k_col_delta(const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
                                                   int64_t n, int16_t *__restrict__ delta, unsigned *__restrict__ wide)
{
    __shared__ int64_t s_rp[257];
    const int64_t r0 = (int64_t)blockIdx.x * 256;
    const int nr = (int)(n - r0 < 256 ? n - r0 : 256);
    for (int t = threadIdx.x; t <= nr; t += 256) s_rp[t] = row_ptr[r0 + t];
    __syncthreads();
    const int64_t e1 = s_rp[nr];
    bool w = false;
    for (int64_t e = s_rp[0] + threadIdx.x; e < e1; e += 256) {
        // the row of e: the last of the block's rows that starts at or before
        // e (an empty row shares its start with the next row)
        int lo = 0, hi = nr - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_rp[mid] <= e) lo = mid; else hi = mid - 1;
        }
        const int64_t d = (int64_t)col[e] - (r0 + lo);
        w |= d < INT16_MIN || d > INT16_MAX;
        delta[e] = (int16_t)d;
    }
    if (__ballot(w) != 0 && (threadIdx.x & 63) == 0) atomicOr(wide, 1u);
}

hipError_t launch_col_delta(const int64_t *row_ptr, const int32_t *col, int64_t n, int16_t *delta, unsigned *wide,
                            hipStream_t s)
{
    hipLaunchKernelGGL(k_col_delta, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, row_ptr, col, n, delta, wide);
    return hipGetLastError();
}

__global__ void k_zero_u64(unsigned long long *p, int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < count; t += stride) p[t] = 0;
}

hipError_t launch_zero_u64(unsigned long long *p, int64_t count, hipStream_t s)
{
    hipLaunchKernelGGL(k_zero_u64, dim3((unsigned)grid_for(count)), dim3(256), 0, s, p, count);
    return hipGetLastError();
}

}  // namespace ul
