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

// Work split of the wavefront epoch kernel: wave w owns the whole rows
// [part[w], part[w+1]); consecutive waves cover about kWaveCost units of
// (edges + row_weight * rows).
constexpr int kWaveCost = 512;
__host__ __device__ constexpr int row_weight(int dim) { return dim > 2 ? dim : 2; }
__host__ __device__ constexpr int rows_cap(int dim) { return kWaveCost / row_weight(dim) + 1; }

// ---- ingest (kernels_prep.hip) ----
struct PrepBuffers {
    // inputs (device)
    const int32_t *rows;
    const int32_t *cols;
    const float *vals;
    int64_t nnz;
    int64_t n;
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
hipError_t launch_partition(const int64_t *row_ptr, int64_t n, int32_t dim, int32_t *part, int64_t n_waves,
                            hipStream_t s);
hipError_t launch_zero_u64(unsigned long long *p, int64_t count, hipStream_t s);

// ---- layout (kernels_layout.hip) ----
hipError_t launch_init(float *E, int64_t n, int32_t dim, uint64_t seed, hipStream_t s);
hipError_t launch_epoch(int kernel, int32_t dim, const EpochArgs &A, const int64_t *row_ptr, const int32_t *col,
                        const float *eps, const int32_t *part, int64_t n_waves, hipStream_t s);
hipError_t launch_debug_active(const float *eps, int64_t nnz, int32_t epoch, uint8_t *out, hipStream_t s);
hipError_t launch_debug_negatives(uint32_t n, uint64_t seed, int32_t epoch, int64_t e_first, int64_t count,
                                  int32_t neg_rate, uint32_t *out, hipStream_t s);
hipError_t launch_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t s);

// ---- fuzzy graph (kernels_graph.hip) ----
hipError_t launch_fuzzy_graph(int64_t n, int32_t k, const int32_t *ids, const float *dists, int32_t *rows,
                              int32_t *cols, float *vals, double *rho, double *sigma, double *partial,
                              int64_t npartial, unsigned *flags, hipStream_t s);
int64_t graph_partials(int64_t n, int32_t k);

}  // namespace ul
