// internal.hpp -- launchers shared between the host API and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layout_device.hpp"

namespace ul {

// Sets the thread-local message read by umap_layout_last_error; returns code.
int set_error(int code, const char *msg);

// Flags raised by the ingest kernels.
enum PrepFlag : unsigned {
    kBadIndex = 1u,
    kBadValue = 2u,
    kDuplicate = 4u,
    kAsymmetric = 8u,
};

// Device-resident scalars of the ingest.
struct PrepScalars {
    unsigned flags;
    unsigned wmax_bits;   // bits of the largest kept candidate weight (> 0)
    int max_degree;
    int pad;
};

// Work split of the wavefront epoch kernels: wave w owns the whole rows
// [part[w], part[w+1]), chosen so that consecutive waves cover about C units
// of (edges + row_weight * rows), C = wave_cost(total units) <= kWaveCost.  The
// row weight bounds the rows of a wave (and so its LDS accumulator) by
// rows_cap; long waves amortise the per-wave set-up and commit, and C shrinks
// (by halves, down to kMinWaveCost) until a graph gives at least
// kTargetWaves waves, so that small graphs still fill the chip.
constexpr int kWaveCost = 8192;
constexpr int kMinWaveCost = 256;
constexpr int64_t kTargetWaves = 4096;
__host__ __device__ constexpr int row_weight(int dim) { return 32 * (dim > 2 ? dim : 2); }
__host__ __device__ constexpr int rows_cap(int dim) { return kWaveCost / row_weight(dim) + 1; }
inline int64_t wave_cost(int64_t total_units)
{
    int64_t c = kWaveCost;
    while (c > kMinWaveCost && total_units / c < kTargetWaves) c >>= 1;
    return c;
}
// Most waves any graph of at most `total_units` gets (wave_cost grows with the
// total, so a smaller total never needs more than 2 kTargetWaves).
inline int64_t max_wave_count(int64_t total_units)
{
    const int64_t big = total_units / kWaveCost;
    return (big > 2 * kTargetWaves ? big : 2 * kTargetWaves) + 2;
}

// ---- ingest (kernels_prep.hip) ----
struct PrepBuffers {
    // inputs (device)
    const int32_t *rows;
    const int32_t *cols;
    const float *vals;
    int64_t nnz;
    int64_t n;          // rows
    int64_t n_cols;     // columns are in [0, n_cols); n unless bipartite
    bool bipartite;     // rows and columns are different vertex sets (no self loops, no symmetry)
    int32_t n_epochs;
    // scratch (device, capacity nnz or n)
    int32_t *deg;       // n
    int32_t *cursor;    // n
    int32_t *trow;      // nnz
    int32_t *tcol;      // nnz
    float *tval;        // nnz
    float *sval;        // nnz, values in sorted order
    int64_t *bsum;      // scan partials
    int64_t nblocks_scan;
    PrepScalars *scalars;
    // outputs (device)
    int64_t *row_ptr;   // n + 1
    int32_t *col;       // nnz (capacity)
    float *eps;         // nnz (capacity)
};

int64_t scan_blocks(int64_t n);
hipError_t launch_prep(const PrepBuffers &B, hipStream_t s);
// Waves over rows [r0, r1) (0 <= r0 < r1); n_waves = ceil(units / cost) for
// the units (edges + row_weight x rows) of the range.
hipError_t launch_partition(const int64_t *row_ptr, int64_t r0, int64_t r1, int32_t dim, int64_t cost,
                            int32_t *part, int64_t n_waves, uint8_t *head, hipStream_t s);
hipError_t launch_zero_u64(unsigned long long *p, int64_t count, hipStream_t s);
// delta[e] = col[e] - row(e) as int16 for the n rows; *wide = 1 (it must start
// at 0) when some delta needs more than 16 bits.
hipError_t launch_col_delta(const int64_t *row_ptr, const int32_t *col, int64_t n, int16_t *delta, unsigned *wide,
                            hipStream_t s);

// ---- layout (kernels_layout.hip) ----
hipError_t launch_init(float *E, int64_t n, int32_t dim, uint64_t seed, hipStream_t s);
hipError_t launch_init_transform(const int64_t *row_ptr, const int32_t *col, const float *eps, const float *T,
                                 int64_t n, int32_t dim, float *E, hipStream_t s);
// Graph-side arrays of the epoch kernels.
struct WaveGraph {
    const int64_t *row_ptr;   // n + 1
    const int32_t *col;       // kept edges, sorted by (row, col)
    const float *eps;         // epochs per sample of each edge
    const uint8_t *head;      // row of each edge relative to its wave's first row
    const int32_t *part;      // n_waves + 1 wave boundaries (rows)
    int64_t n_waves;
    // negative samples are filed by vertex-table range: P = 2^lg_phases ranges
    int32_t n_phases;
    int32_t lg_phases;
    uint32_t *rec;            // records ((row in wave) << 24 | offset in range), slots by record_offset
    int32_t *rec_count;       // P x n_waves
    unsigned *overflow;       // set when a record did not fit its range slot
    int64_t cap_limit;        // < 0: none; else record slots per range are cut to it (failure injection)
    long long *delta;         // n x dim fixed-point partial sums between launches
    const int16_t *col16;     // col - row in 16 bits when every edge's fits (a fit), else null
};

// First record slot of wave w (edges from e0): every wave gets
// 1.25 x neg_rate x its edges + 256 x P slots, split evenly over the P table
// ranges.  A range of a wave gets more than its share of a wave's draws only
// with vanishing probability (the ranges split uniform random words); a draw
// that finds its range full raises the overflow flag and the epochs are redone
// by the one-thread-per-vertex kernel.
__host__ __device__ inline int64_t record_offset(int64_t w, int64_t e0, int32_t neg_rate, int32_t n_phases)
{
    return (5 * (int64_t)neg_rate * e0 + 3) / 4 + (int64_t)256 * n_phases * w;
}

// At most this many table ranges (phases) per epoch.
constexpr int kMaxPhases = 16;
// The range count trades the gathers' L2 hit rate (a range of about 2 MB
// stays resident in one XCD's 4 MB L2 next to the streamed edge data) against
// the cost of each further range: one more launch and one more round trip of
// the n x dim int64 partial sums.  Measured on 1M and 5M vertices with 2 to 16
// components, the best count is 4 up to about 2.5M vertices and 8 at 5M,
// whatever the row width, and never more than a 2 MB range needs.
constexpr int64_t kPhaseTableBytes = 2 << 20;
constexpr int64_t kPhaseRows = 2500000;
// With one range the draw kernel applies the repulsions itself (no records,
// no partial sums, one launch per epoch), which beats the range launches for
// tables up to kOneRangeBytes (200 epochs of window graphs, ms, one range
// against the split: 2 components 700K vertices 37.3 / 45.5; 3 components 500K
// 32.6 / 38.1; 4 components 350K 26.3 / 31.3; 8 components 180K 27.8 / 28.1),
// and up to kOneRangeBytesWide from 9 to kOneRangeMaxDim components (10
// components 100K 21.2 / 21.5, 12 components 80K 18.5 / 19.0, 13 components
// 75K 19.0 / 19.3).  Wider rows keep the plain rule (one range up to 2 MB):
// 14 components 70K 19.7 / 19.4, 16 components 60K / 45K / 35K 20.0 / 18.9,
// 15.6 / 15.1, 13.2 / 13.0.
constexpr int64_t kOneRangeBytes = 6 << 20;
constexpr int64_t kOneRangeBytesWide = 4 << 20;
constexpr int32_t kOneRangeMaxDim = 13;
// log2 of the number of ranges for a table of n vertices x dim: 0 up to
// kOneRangeBytes (kOneRangeBytesWide from 9 to kOneRangeMaxDim components);
// else min(the ranges that bring a range down to kPhaseTableBytes, 4 ranges per
// kPhaseRows vertices rounded up to a power of two), at most kMaxPhases.
int32_t phase_log2(int64_t n, int32_t dim);

hipError_t launch_epoch(int kernel, int32_t dim, const EpochArgs &A, const WaveGraph &G, hipStream_t s);
// One asynchronous epoch, in place on A.E_next (A.E must be the same buffer).
hipError_t launch_epoch_hogwild(int32_t dim, const EpochArgs &A, const WaveGraph &G, hipStream_t s);
// Count slots one epoch of `kernel` writes (one per wave).
int64_t count_slots(int kernel, int64_t n, int64_t n_waves);
// out[r] = sum of counts[r * stride + 0 .. slots) for r < rows.
hipError_t launch_reduce_counts(const int32_t *counts, int64_t stride, int64_t slots, int32_t rows,
                                unsigned long long *out, hipStream_t s);
// *out = a[0] + ... + a[n - 1].
hipError_t launch_sum_u64(const unsigned long long *a, int64_t n, unsigned long long *out, hipStream_t s);
// Epochs whose per-wave counts are kept before they are summed.
constexpr int kCountRing = 256;
hipError_t launch_debug_active(const float *eps, int64_t nnz, int32_t epoch, uint8_t *out, hipStream_t s);
hipError_t launch_debug_negatives(uint32_t n, uint64_t seed, int32_t epoch, int64_t e_first, int64_t count,
                                  int32_t neg_rate, uint32_t *out, hipStream_t s);
hipError_t launch_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t s);
hipError_t launch_probe_gather(const void *table, int64_t entries, int64_t threads, int32_t iters, void *out,
                               hipStream_t s);

// ---- trustworthiness (kernels_trust.hip) ----
// Scratch: nx[n], nbr[n k], thr[n k], cnt[n k], pen[n], sum[1], flags[1]
// (flags zeroed by the caller).
hipError_t launch_trustworthiness(const float *X, int64_t n, int32_t d, const float *Y, int32_t dim, int32_t k,
                                  float *nx, int32_t *nbr, float *thr, int32_t *cnt, int64_t *pen,
                                  unsigned long long *sum, unsigned *flags, hipStream_t s);

// ---- fuzzy graph (kernels_graph.hip) ----
hipError_t launch_fuzzy_graph(int64_t n, int32_t k, const int32_t *ids, const float *dists, int32_t *rows,
                              int32_t *cols, float *vals, double *rho, double *sigma, double *partial,
                              int64_t npartial, unsigned *flags, hipStream_t s);
int64_t graph_partials(int64_t n, int32_t k);

}  // namespace ul
