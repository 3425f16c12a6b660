// api.hip -- host side of the C ABI declared in include/umap_layout.h.
//
// Argument checks that need no GPU run first; then one device arena holds
// everything the handle keeps (CSR graph, wave partition, two embedding
// buffers for the epoch-synchronous ping-pong, per-epoch counters), and a
// stream-ordered scratch allocation holds the ingest's temporaries.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "umap_layout.h"
#include "internal.hpp"

namespace {

thread_local std::string g_err;

__attribute__((format(printf, 2, 3))) int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

struct HipFailure {
    hipError_t err;
    const char *what;
};

#define UL_HIP(expr)                                    \
    do {                                                \
        hipError_t ul_e_ = (expr);                      \
        if (ul_e_ != hipSuccess) throw HipFailure{ul_e_, #expr}; \
    } while (0)

int hip_fail(const HipFailure &f)
{
    if (f.err == hipErrorOutOfMemory || f.err == hipErrorMemoryAllocation)
        return fail(UMAP_E_NOMEM, "device allocation failed (%s): %s", f.what, hipGetErrorString(f.err));
    return fail(UMAP_E_DEVICE, "HIP call failed (%s): %s", f.what, hipGetErrorString(f.err));
}

// Optional failure injection for tests: UMAP_LAYOUT_FAULT=alloc makes the
// arena allocation report out-of-memory; UMAP_LAYOUT_FAULT=launch@K makes the
// launch of epoch K report a device error (nothing is launched in either
// case); UMAP_LAYOUT_FAULT=records gives the wavefront kernel no record slots,
// so every negative sample overflows and the epochs are redone.
bool fault_alloc()
{
    const char *f = getenv("UMAP_LAYOUT_FAULT");
    return f && strcmp(f, "alloc") == 0;
}

bool fault_records()
{
    const char *f = getenv("UMAP_LAYOUT_FAULT");
    return f && strcmp(f, "records") == 0;
}

int fault_launch_epoch()
{
    const char *f = getenv("UMAP_LAYOUT_FAULT");
    if (!f || strncmp(f, "launch@", 7) != 0) return -1;
    return atoi(f + 7);
}

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

struct Carver {
    char *base;
    size_t off = 0;
    template <typename T>
    T *take(size_t count)
    {
        T *p = reinterpret_cast<T *>(base + off);
        off += align_up(count * sizeof(T) > 0 ? count * sizeof(T) : 1);
        return p;
    }
};

template <typename T>
size_t need(size_t count)
{
    return align_up(count * sizeof(T) > 0 ? count * sizeof(T) : 1);
}

int check_scalars(int64_t n, int32_t dim, int64_t nnz, float a, float b, int32_t n_epochs, int32_t neg_rate)
{
    if (n < 1 || n >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "n must be in [1, 2^31), got %lld", (long long)n);
    if (dim < 1 || dim > 16) return fail(UMAP_E_INVAL, "n_components must be in [1, 16], got %d", dim);
    if (nnz < 0 || nnz >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "nnz must be in [0, 2^31), got %lld", (long long)nnz);
    if (!(a > 0.0f) || !isfinite(a)) return fail(UMAP_E_INVAL, "a must be a positive finite value");
    if (!(b > 0.0f) || !isfinite(b)) return fail(UMAP_E_INVAL, "b must be a positive finite value");
    if (n_epochs < 1 || n_epochs >= (1 << 24)) return fail(UMAP_E_INVAL, "n_epochs must be in [1, 2^24), got %d", n_epochs);
    if (neg_rate < 0 || neg_rate >= (1 << 16)) return fail(UMAP_E_INVAL, "neg_rate must be in [0, 2^16), got %d", neg_rate);
    return UMAP_OK;
}

}  // namespace

int ul::set_error(int code, const char *msg)
{
    g_err = msg;
    return code;
}

struct umap_layout {
    int device = 0;
    hipStream_t stream = nullptr;
    int64_t n = 0;
    int32_t dim = 0;
    float a = 0, b = 0;
    int32_t n_epochs = 0, neg_rate = 0;
    int64_t nnz_in = 0, nnz = 0;
    int32_t max_degree = 0;
    float w_max = 0;
    int kernel = 0;
    int mode = 0;                           // 0 epoch-synchronous, 1 asynchronous in place
    float *table = nullptr;                 // transform: the frozen layout (n_table x dim), else null
    int64_t n_table = 0;                    // rows of the table the tails and negatives index

    void *arena = nullptr;
    int64_t *row_ptr = nullptr;
    int32_t *col = nullptr;
    int16_t *col16 = nullptr;               // col - row in 16 bits (a fit whose deltas all fit)
    bool col16_ok = false;
    float *eps = nullptr;
    int32_t *part = nullptr;
    int64_t n_waves = 0;
    int64_t max_waves = 0;                  // capacity of part, rec_count and the record slots
    int64_t row_first = 0, row_last = 0;    // rows the epochs update (umap_layout_set_rows)
    uint8_t *head = nullptr;       // edge's row relative to its wave's first row
    float *E[2] = {nullptr, nullptr};
    int cur = 0;
    bool has_layout = false;
    unsigned long long *active = nullptr;   // n_epochs sampled-edge counts
    unsigned long long *active_sum = nullptr;   // their sum over the last call's epochs
    int32_t *counts = nullptr;              // ring of per-wave counts
    int32_t lg_phases = 0;                  // negative samples split over 2^lg table ranges
    uint32_t *rec = nullptr;                // records of negative samples, slots by record_offset
    unsigned *overflow = nullptr;           // raised when a record slot was full
    float *E_start = nullptr;               // layout at the start of a call, for a redo
    int32_t *rec_count = nullptr;           // per range and wave
    long long *delta = nullptr;             // fixed-point partial sums between launches
    int64_t count_stride = 0;               // slots per ring row
    hipEvent_t ev[3] = {nullptr, nullptr, nullptr};
    bool time_epochs = false;               // umap_layout_set_epoch_timing
    std::vector<hipEvent_t> ep_ev;          // per-epoch events (created on first use)
    int32_t timed = 0;                      // epochs the last call timed
    umap_layout_stats_t st{};

    void release()
    {
        if (stream || arena) (void)hipStreamSynchronize(stream);
        for (auto &e : ev)
            if (e) (void)hipEventDestroy(e);
        for (auto &e : ep_ev)
            if (e) (void)hipEventDestroy(e);
        ep_ev.clear();
        if (arena) (void)hipFree(arena);
        arena = nullptr;
    }
};

namespace {

// A fit (table == nullptr: B is symmetric over n vertices) or a transform
// (rows are n new points, columns index the n_table rows of the frozen host
// layout `table`).
int create_common(umap_layout **out, int64_t n, int32_t dim, const int32_t *rows, const int32_t *cols,
                  const float *vals, int64_t nnz, float a, float b, int32_t n_epochs, int32_t neg_rate,
                  hipStream_t stream, bool host_inputs, const float *table = nullptr, int64_t n_table = 0)
{
    umap_layout *h = new (std::nothrow) umap_layout();
    if (!h) return fail(UMAP_E_NOMEM, "host allocation failed");
    void *scratch = nullptr;
    try {
        int ndev = 0;
        if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
            delete h;
            return fail(UMAP_E_DEVICE, "no HIP device available");
        }
        UL_HIP(hipGetDevice(&h->device));
        h->stream = stream;
        h->n = n;
        h->dim = dim;
        h->a = a;
        h->b = b;
        h->n_epochs = n_epochs;
        h->neg_rate = neg_rate;
        h->nnz_in = nnz;
        h->n_table = table ? n_table : n;
        h->row_first = 0;
        h->row_last = n;
        for (auto &e : h->ev) UL_HIP(hipEventCreate(&e));

        // persistent arena; the wave count is bounded with nnz (kept <= nnz)
        const int wgt = ul::row_weight(dim);
        const int64_t max_waves = ul::max_wave_count(nnz + (int64_t)wgt * n);
        h->max_waves = max_waves;
        const size_t nd = (size_t)n * (size_t)dim;
        const int64_t count_stride =
            ul::count_slots(1, n, 0) > max_waves ? ul::count_slots(1, n, 0) : max_waves;
        const int64_t count_rows = n_epochs < ul::kCountRing ? n_epochs : ul::kCountRing;
        const int32_t lg_phases = ul::phase_log2(h->n_table, dim);
        const size_t table_elems = table ? (size_t)n_table * (size_t)dim : 0;
        const int64_t n_phases = (int64_t)1 << lg_phases;
        size_t bytes = need<int64_t>(n + 1) + need<int32_t>(nnz) + need<int16_t>(table ? 0 : nnz) + need<float>(nnz) +
                       need<int32_t>(max_waves + 1) +
                       2 * need<float>(nd) + need<unsigned long long>(n_epochs) + need<unsigned long long>(1) +
                       need<uint8_t>(nnz) +
                       need<int32_t>((size_t)count_rows * count_stride) +
                       need<uint32_t>(ul::record_offset(max_waves, nnz, neg_rate, (int32_t)n_phases)) +
                       need<int32_t>((size_t)n_phases * max_waves) + need<long long>(nd) + need<unsigned>(1) +
                       need<float>(nd) + need<float>(table_elems);
        if (fault_alloc()) throw HipFailure{hipErrorOutOfMemory, "hipMalloc(arena) [injected]"};
        UL_HIP(hipMalloc(&h->arena, bytes));
        Carver cv{static_cast<char *>(h->arena)};
        h->row_ptr = cv.take<int64_t>(n + 1);
        h->col = cv.take<int32_t>(nnz);
        h->col16 = cv.take<int16_t>(table ? 0 : nnz);
        h->eps = cv.take<float>(nnz);
        h->part = cv.take<int32_t>(max_waves + 1);
        h->E[0] = cv.take<float>(nd);
        h->E[1] = cv.take<float>(nd);
        h->active = cv.take<unsigned long long>(n_epochs);
        h->active_sum = cv.take<unsigned long long>(1);
        h->head = cv.take<uint8_t>(nnz);
        h->counts = cv.take<int32_t>((size_t)count_rows * count_stride);
        h->count_stride = count_stride;
        h->lg_phases = lg_phases;
        h->rec = cv.take<uint32_t>(ul::record_offset(max_waves, nnz, neg_rate, (int32_t)n_phases));
        h->rec_count = cv.take<int32_t>((size_t)n_phases * max_waves);
        h->delta = cv.take<long long>(nd);
        h->overflow = cv.take<unsigned>(1);
        h->E_start = cv.take<float>(nd);
        if (table) {
            h->table = cv.take<float>(table_elems);
            UL_HIP(hipMemcpyAsync(h->table, table, sizeof(float) * table_elems, hipMemcpyHostToDevice, stream));
        }

        // ingest scratch (stream-ordered)
        ul::PrepBuffers B{};
        B.nnz = nnz;
        B.n = n;
        B.n_cols = h->n_table;
        B.bipartite = table != nullptr;
        B.n_epochs = n_epochs;
        B.nblocks_scan = ul::scan_blocks(n);
        size_t sbytes = 2 * need<int32_t>(n) + 2 * need<int32_t>(nnz) + 2 * need<float>(nnz) +
                        need<int64_t>(B.nblocks_scan) + need<ul::PrepScalars>(1);
        if (host_inputs) sbytes += 2 * need<int32_t>(nnz) + need<float>(nnz);
        UL_HIP(hipMallocAsync(&scratch, sbytes, stream));
        Carver sc{static_cast<char *>(scratch)};
        B.deg = sc.take<int32_t>(n);
        B.cursor = sc.take<int32_t>(n);
        B.trow = sc.take<int32_t>(nnz);
        B.tcol = sc.take<int32_t>(nnz);
        B.tval = sc.take<float>(nnz);
        B.sval = sc.take<float>(nnz);
        B.bsum = sc.take<int64_t>(B.nblocks_scan);
        B.scalars = sc.take<ul::PrepScalars>(1);
        if (host_inputs) {
            int32_t *dr = sc.take<int32_t>(nnz);
            int32_t *dc = sc.take<int32_t>(nnz);
            float *dv = sc.take<float>(nnz);
            if (nnz) {
                UL_HIP(hipMemcpyAsync(dr, rows, sizeof(int32_t) * nnz, hipMemcpyHostToDevice, stream));
                UL_HIP(hipMemcpyAsync(dc, cols, sizeof(int32_t) * nnz, hipMemcpyHostToDevice, stream));
                UL_HIP(hipMemcpyAsync(dv, vals, sizeof(float) * nnz, hipMemcpyHostToDevice, stream));
            }
            B.rows = dr;
            B.cols = dc;
            B.vals = dv;
        } else {
            B.rows = rows;
            B.cols = cols;
            B.vals = vals;
        }
        B.row_ptr = h->row_ptr;
        B.col = h->col;
        B.eps = h->eps;

        UL_HIP(hipEventRecord(h->ev[0], stream));
        UL_HIP(hipMemsetAsync(B.deg, 0, 2 * need<int32_t>(n), stream));   // deg and cursor are adjacent
        UL_HIP(hipMemsetAsync(B.scalars, 0, sizeof(ul::PrepScalars), stream));
        UL_HIP(ul::launch_prep(B, stream));
        UL_HIP(hipEventRecord(h->ev[1], stream));

        ul::PrepScalars S{};
        int64_t kept = 0;
        UL_HIP(hipMemcpyAsync(&S, B.scalars, sizeof S, hipMemcpyDeviceToHost, stream));
        UL_HIP(hipMemcpyAsync(&kept, h->row_ptr + n, sizeof kept, hipMemcpyDeviceToHost, stream));
        UL_HIP(hipStreamSynchronize(stream));
        UL_HIP(hipFreeAsync(scratch, stream));
        scratch = nullptr;

        int rc = UMAP_OK;
        if (S.flags & ul::kBadIndex)
            rc = table ? fail(UMAP_E_INVAL, "a row index is outside [0, n_new) or a column outside [0, n_table)")
                       : fail(UMAP_E_INVAL, "a row or column index is outside [0, n)");
        else if (S.flags & ul::kBadValue) rc = fail(UMAP_E_INVAL, "a value is not finite");
        else if (S.flags & ul::kDuplicate) rc = fail(UMAP_E_INVAL, "an edge (i, j) is listed more than once");
        else if (S.flags & ul::kAsymmetric)
            rc = fail(UMAP_E_ASYMMETRIC, "the graph is not symmetric: a kept (i, j, v) has no (j, i) with equal v");
        else if ((int64_t)S.max_degree * (8 + 4 * (int64_t)neg_rate) >= ((int64_t)1 << 31))
            rc = fail(UMAP_E_INVAL, "a row of %d edges is too long for the fixed-point accumulator", S.max_degree);
        if (rc != UMAP_OK) {
            h->release();
            delete h;
            return rc;
        }
        h->nnz = kept;
        h->max_degree = S.max_degree;
        memcpy(&h->w_max, &S.wmax_bits, sizeof(float));
        const int64_t units = kept + (int64_t)wgt * n;
        const int64_t cost = ul::wave_cost(units);
        h->n_waves = (units + cost - 1) / cost;
        if (h->n_waves < 1) h->n_waves = 1;
        if (h->n_waves > max_waves) throw HipFailure{hipErrorInvalidValue, "wave count exceeds the arena"};
        UL_HIP(ul::launch_partition(h->row_ptr, 0, n, dim, cost, h->part, h->n_waves, h->head, stream));
        if (!table && kept > 0) {
            // a fit's tails as 16-bit offsets from their rows, where they all fit
            unsigned wide = 1;
            UL_HIP(hipMemsetAsync(h->overflow, 0, sizeof(unsigned), stream));
            UL_HIP(ul::launch_col_delta(h->row_ptr, h->col, n, h->col16, h->overflow, stream));
            UL_HIP(hipMemcpyAsync(&wide, h->overflow, sizeof wide, hipMemcpyDeviceToHost, stream));
            UL_HIP(hipStreamSynchronize(stream));
            h->col16_ok = wide == 0;
        }
        float ms = 0;
        UL_HIP(hipEventElapsedTime(&ms, h->ev[0], h->ev[1]));
        h->st.prep_ms = ms;
        *out = h;
        return UMAP_OK;
    } catch (const HipFailure &f) {
        int rc = hip_fail(f);
        if (scratch) (void)hipFreeAsync(scratch, stream);
        h->release();
        delete h;
        return rc;
    } catch (...) {
        if (scratch) (void)hipFreeAsync(scratch, stream);
        h->release();
        delete h;
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int run_epochs_impl(umap_layout *h, uint64_t seed, int32_t first, int32_t last, bool timed_init)
{
    const int fault = fault_launch_epoch();
    ul::EpochArgs A{};
    A.n = (uint32_t)h->n;
    A.row_first = (uint32_t)h->row_first;
    A.row_last = (uint32_t)h->row_last;
    A.n_table = (uint32_t)h->n_table;
    A.same_table = h->table ? 0 : 1;
    A.attr_mult = h->table ? 1.0f : 2.0f;
    A.neg_rate = h->neg_rate;
    A.a = h->a;
    A.b = h->b;
    A.key_lo = (uint32_t)seed;
    A.key_hi = (uint32_t)(seed >> 32);
    ul::WaveGraph G{h->row_ptr,     h->col,       h->eps,    h->head,      h->part,
                    h->n_waves,     1 << h->lg_phases,       h->lg_phases, h->rec,
                    h->rec_count,   h->overflow,  fault_records() ? (int64_t)0 : (int64_t)-1,
                    h->delta,       h->col16_ok ? h->col16 : nullptr};
    // the wave kernels store a sample's offset inside its table range and a
    // sampled edge's offset inside its wave in 24 bits (a wave holds fewer
    // than kWaveCost + max_degree edges), and address a wave's record slots
    // (1.25 neg_rate x its edges + 256 P) by 32-bit byte offsets; beyond that
    // (n >= 2^28 vertices, a row of about 2^24 edges, or a huge neg_rate) the
    // one-thread-per-vertex kernel runs
    const int64_t wave_slots = (5 * (int64_t)h->neg_rate * ((int64_t)ul::kWaveCost + h->max_degree) + 3) / 4 +
                               (int64_t)256 * (1 << h->lg_phases) + 1;
    const bool fits = (h->n_table >> h->lg_phases) + 2 < ((int64_t)1 << 24) &&
                      (int64_t)h->max_degree + ul::kWaveCost < ((int64_t)1 << 24) &&
                      wave_slots * (int64_t)sizeof(uint32_t) < ((int64_t)1 << 32);
    const bool async = h->mode == 1;
    if (async && h->table) return fail(UMAP_E_INVAL, "the asynchronous mode applies to fits, not to transforms");
    const bool restricted = h->row_first > 0 || h->row_last < h->n;
    if (async && restricted) return fail(UMAP_E_INVAL, "the asynchronous mode updates all rows (umap_layout_set_rows)");
    // epoch kernel: 0 edge-parallel, 1 one thread per vertex, kAsyncKernel the
    // per-edge asynchronous kernel.  In the asynchronous mode kernel 0 runs in
    // place (each launch adds its sums to the rows it owns) and kernel 1
    // chooses the per-edge kernel, which is also taken where the 24-bit
    // offsets of kernel 0 do not fit.
    constexpr int kAsyncKernel = -1;
    const int kernel = async ? (fits && h->kernel == 0 ? 0 : kAsyncKernel) : fits ? h->kernel : 1;
    if (kernel == kAsyncKernel && (int64_t)h->max_degree + ul::kWaveCost >= ((int64_t)1 << 24))
        return fail(UMAP_E_INVAL, "the per-edge asynchronous kernel needs rows of fewer than %d edges",
                    (1 << 24) - ul::kWaveCost);
    // with one table range the draw kernel applies every negative itself and
    // files no records, so no slot can overflow and no redo is needed
    const bool records = kernel == 0 && h->lg_phases > 0;
    const int cur0 = h->cur;
    const size_t row_bytes = sizeof(float) * (size_t)h->dim;
    const size_t nd_bytes = row_bytes * (size_t)h->n;
    if (restricted && !async) {
        // rows outside the range are not written by the epochs: make both
        // buffers hold them, so that they keep their values
        float *src = h->E[cur0], *dst = h->E[1 - cur0];
        if (h->row_first > 0)
            UL_HIP(hipMemcpyAsync(dst, src, row_bytes * (size_t)h->row_first, hipMemcpyDeviceToDevice, h->stream));
        if (h->row_last < h->n)
            UL_HIP(hipMemcpyAsync(dst + (size_t)h->row_last * h->dim, src + (size_t)h->row_last * h->dim,
                                  row_bytes * (size_t)(h->n - h->row_last), hipMemcpyDeviceToDevice, h->stream));
    }
    if (records) {
        // the layout this call starts from, in case a record slot overflows
        UL_HIP(hipMemsetAsync(h->overflow, 0, sizeof(unsigned), h->stream));
        UL_HIP(hipMemcpyAsync(h->E_start, h->E[cur0], nd_bytes, hipMemcpyDeviceToDevice, h->stream));
    }
    UL_HIP(hipEventRecord(h->ev[1], h->stream));

    // per-epoch events: one before each of the first UMAP_MAX_TIMED_EPOCHS
    // epochs of the call and one after the last of them
    h->timed = 0;
    const int32_t timed = h->time_epochs ? (last - first < UMAP_MAX_TIMED_EPOCHS ? last - first : UMAP_MAX_TIMED_EPOCHS)
                                         : 0;
    if (timed > 0) {
        while ((int32_t)h->ep_ev.size() < timed + 1) {
            hipEvent_t e = nullptr;
            UL_HIP(hipEventCreate(&e));
            h->ep_ev.push_back(e);
        }
    }
    // epochs [first, last) with one kernel; fault >= 0 injects a launch error
    auto epochs = [&](int which) -> int {
        UL_HIP(ul::launch_zero_u64(h->active, h->n_epochs, h->stream));
        const int64_t slots = ul::count_slots(which == 1 ? 1 : 0, h->row_last - h->row_first, h->n_waves);
        const int ring = h->n_epochs < ul::kCountRing ? h->n_epochs : ul::kCountRing;
        int32_t pending_from = first;   // first epoch whose counts are not yet summed
        for (int32_t ep = first; ep < last; ++ep) {
            if (ep == fault) {
                UL_HIP(hipStreamSynchronize(h->stream));
                return fail(UMAP_E_DEVICE, "epoch %d launch failed [injected]", ep);
            }
            if (ep - first < timed) UL_HIP(hipEventRecord(h->ep_ev[(size_t)(ep - first)], h->stream));
            A.epoch = ep;
            A.alpha = 1.0 - (double)ep / (double)h->n_epochs;
            A.counts = h->counts + (int64_t)((ep - pending_from) % ring) * h->count_stride;
            if (which == kAsyncKernel) {
                A.E = A.E_next = h->E[h->cur];   // in place
                A.T = A.E;
                UL_HIP(ul::launch_epoch_hogwild(h->dim, A, G, h->stream));
            } else {
                A.E = h->E[h->cur];
                A.E_next = h->E[async ? h->cur : 1 - h->cur];
                A.in_place = async ? 1 : 0;
                A.T = h->table ? h->table : A.E;
                UL_HIP(ul::launch_epoch(which, h->dim, A, G, h->stream));
                if (!async) h->cur = 1 - h->cur;
            }
            if (ep + 1 - first == timed) UL_HIP(hipEventRecord(h->ep_ev[(size_t)timed], h->stream));
            if (ep + 1 - pending_from == ring || ep + 1 == last) {
                UL_HIP(ul::launch_reduce_counts(h->counts, h->count_stride, slots, ep + 1 - pending_from,
                                                h->active + pending_from, h->stream));
                pending_from = ep + 1;
            }
        }
        return UMAP_OK;
    };

    int rc = epochs(kernel);
    if (rc != UMAP_OK) return rc;
    h->st.overflow_redone = 0;
    if (records) {
        unsigned overflow = 0;
        UL_HIP(hipMemcpyAsync(&overflow, h->overflow, sizeof overflow, hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipStreamSynchronize(h->stream));
        if (overflow) {
            // a range slot was full: some negative samples were not applied;
            // redo the call's epochs from its starting layout with the
            // one-thread-per-vertex kernel, which keeps no records (in place
            // in the asynchronous mode)
            h->cur = cur0;
            UL_HIP(hipMemcpyAsync(h->E[cur0], h->E_start, nd_bytes, hipMemcpyDeviceToDevice, h->stream));
            rc = epochs(1);
            if (rc != UMAP_OK) return rc;
            h->st.overflow_redone = 1;
        }
    }
    UL_HIP(hipEventRecord(h->ev[2], h->stream));
    // the call's sampled-edge count, summed on the device (8 bytes come back)
    unsigned long long total = 0;
    UL_HIP(ul::launch_sum_u64(h->active + first, last - first, h->active_sum, h->stream));
    UL_HIP(hipMemcpyAsync(&total, h->active_sum, sizeof total, hipMemcpyDeviceToHost, h->stream));
    UL_HIP(hipStreamSynchronize(h->stream));
    float ms = 0;
    UL_HIP(hipEventElapsedTime(&ms, h->ev[1], h->ev[2]));
    h->st.epochs_ms = ms;
    if (timed_init) {
        UL_HIP(hipEventElapsedTime(&ms, h->ev[0], h->ev[1]));
        h->st.init_ms = ms;
    }
    h->st.epochs_done = last - first;
    h->timed = timed;
    h->st.active_edges = (int64_t)total;
    h->st.edge_updates = (int64_t)total * (1 + h->neg_rate);
    return UMAP_OK;
}

}  // namespace

extern "C" {

const char *umap_layout_last_error(void) { return g_err.c_str(); }

int umap_layout_create(umap_layout **out, int64_t n, int32_t n_components, const int32_t *rows, const int32_t *cols,
                       const float *vals, int64_t nnz, float a, float b, int32_t n_epochs, int32_t neg_rate)
{
    try {
        if (!out) return fail(UMAP_E_INVAL, "out is NULL");
        *out = nullptr;
        int rc = check_scalars(n, n_components, nnz, a, b, n_epochs, neg_rate);
        if (rc) return rc;
        if (nnz > 0 && (!rows || !cols || !vals)) return fail(UMAP_E_INVAL, "rows, cols and vals must not be NULL");
        for (int64_t t = 0; t < nnz; ++t) {
            if (rows[t] < 0 || rows[t] >= n || cols[t] < 0 || cols[t] >= n)
                return fail(UMAP_E_INVAL, "entry %lld: index (%d, %d) outside [0, %lld)", (long long)t, rows[t],
                            cols[t], (long long)n);
            if (!isfinite(vals[t])) return fail(UMAP_E_INVAL, "entry %lld: value is not finite", (long long)t);
        }
        return create_common(out, n, n_components, rows, cols, vals, nnz, a, b, n_epochs, neg_rate, nullptr, true);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int umap_transform_create(umap_layout **out, int64_t n_new, int32_t n_components, const float *table,
                          int64_t n_table, const int32_t *rows, const int32_t *cols, const float *vals, int64_t nnz,
                          float a, float b, int32_t n_epochs, int32_t neg_rate)
{
    try {
        if (!out) return fail(UMAP_E_INVAL, "out is NULL");
        *out = nullptr;
        int rc = check_scalars(n_new, n_components, nnz, a, b, n_epochs, neg_rate);
        if (rc) return rc;
        if (n_table < 1 || n_table >= ((int64_t)1 << 31))
            return fail(UMAP_E_INVAL, "n_table must be in [1, 2^31), got %lld", (long long)n_table);
        if (!table) return fail(UMAP_E_INVAL, "table is NULL");
        if (nnz > 0 && (!rows || !cols || !vals)) return fail(UMAP_E_INVAL, "rows, cols and vals must not be NULL");
        const size_t table_elems = (size_t)n_table * (size_t)n_components;
        for (size_t t = 0; t < table_elems; ++t)
            if (!isfinite(table[t])) return fail(UMAP_E_INVAL, "table entry %zu is not finite", t);
        for (int64_t t = 0; t < nnz; ++t) {
            if (rows[t] < 0 || rows[t] >= n_new || cols[t] < 0 || cols[t] >= n_table)
                return fail(UMAP_E_INVAL, "entry %lld: index (%d, %d) outside [0, %lld) x [0, %lld)", (long long)t,
                            rows[t], cols[t], (long long)n_new, (long long)n_table);
            if (!isfinite(vals[t])) return fail(UMAP_E_INVAL, "entry %lld: value is not finite", (long long)t);
        }
        return create_common(out, n_new, n_components, rows, cols, vals, nnz, a, b, n_epochs, neg_rate, nullptr,
                             true, table, n_table);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int umap_layout_create_device(umap_layout **out, int64_t n, int32_t n_components, const int32_t *rows,
                              const int32_t *cols, const float *vals, int64_t nnz, float a, float b, int32_t n_epochs,
                              int32_t neg_rate, void *stream)
{
    try {
        if (!out) return fail(UMAP_E_INVAL, "out is NULL");
        *out = nullptr;
        int rc = check_scalars(n, n_components, nnz, a, b, n_epochs, neg_rate);
        if (rc) return rc;
        if (nnz > 0 && (!rows || !cols || !vals)) return fail(UMAP_E_INVAL, "rows, cols and vals must not be NULL");
        return create_common(out, n, n_components, rows, cols, vals, nnz, a, b, n_epochs, neg_rate,
                             static_cast<hipStream_t>(stream), false);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

namespace {

void init_layout(umap_layout *h, uint64_t seed)
{
    if (h->table)
        UL_HIP(ul::launch_init_transform(h->row_ptr, h->col, h->eps, h->table, h->n, h->dim, h->E[h->cur],
                                         h->stream));
    else
        UL_HIP(ul::launch_init(h->E[h->cur], h->n, h->dim, seed, h->stream));
    h->has_layout = true;
}

}  // namespace

int umap_layout_init(umap_layout *h, uint64_t seed)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    try {
        UL_HIP(hipSetDevice(h->device));
        init_layout(h, seed);
        UL_HIP(hipStreamSynchronize(h->stream));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int umap_layout_run(umap_layout *h, uint64_t seed)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    try {
        UL_HIP(hipSetDevice(h->device));
        UL_HIP(hipEventRecord(h->ev[0], h->stream));
        init_layout(h, seed);
        return run_epochs_impl(h, seed, 0, h->n_epochs, true);
    } catch (const HipFailure &f) {
        return hip_fail(f);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int umap_layout_run_epochs(umap_layout *h, uint64_t seed, int32_t first, int32_t last)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    if (first < 0 || first > last || last > h->n_epochs)
        return fail(UMAP_E_INVAL, "need 0 <= first <= last <= n_epochs (%d), got %d, %d", h->n_epochs, first, last);
    if (!h->has_layout) return fail(UMAP_E_STATE, "no layout yet: call umap_layout_run or umap_layout_set_embedding");
    try {
        UL_HIP(hipSetDevice(h->device));
        return run_epochs_impl(h, seed, first, last, false);
    } catch (const HipFailure &f) {
        return hip_fail(f);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int umap_layout_get(const umap_layout *h, float *out)
{
    if (!h || !out) return fail(UMAP_E_INVAL, "handle or out is NULL");
    if (!h->has_layout) return fail(UMAP_E_STATE, "no layout yet");
    try {
        UL_HIP(hipSetDevice(h->device));
        UL_HIP(hipMemcpyAsync(out, h->E[h->cur], sizeof(float) * h->n * h->dim, hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipStreamSynchronize(h->stream));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_layout_get_device(const umap_layout *h, float *dev_out)
{
    if (!h || !dev_out) return fail(UMAP_E_INVAL, "handle or dev_out is NULL");
    if (!h->has_layout) return fail(UMAP_E_STATE, "no layout yet");
    try {
        UL_HIP(hipSetDevice(h->device));
        UL_HIP(hipMemcpyAsync(dev_out, h->E[h->cur], sizeof(float) * h->n * h->dim, hipMemcpyDeviceToDevice,
                              h->stream));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_layout_set_embedding(umap_layout *h, const float *host)
{
    if (!h || !host) return fail(UMAP_E_INVAL, "handle or host is NULL");
    try {
        UL_HIP(hipSetDevice(h->device));
        UL_HIP(hipMemcpyAsync(h->E[h->cur], host, sizeof(float) * h->n * h->dim, hipMemcpyHostToDevice, h->stream));
        UL_HIP(hipStreamSynchronize(h->stream));
        h->has_layout = true;
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_layout_get_graph(const umap_layout *h, int64_t *row_ptr, int32_t *col, float *eps, int64_t *nnz_kept)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    try {
        UL_HIP(hipSetDevice(h->device));
        if (row_ptr)
            UL_HIP(hipMemcpyAsync(row_ptr, h->row_ptr, sizeof(int64_t) * (h->n + 1), hipMemcpyDeviceToHost, h->stream));
        if (col && h->nnz)
            UL_HIP(hipMemcpyAsync(col, h->col, sizeof(int32_t) * h->nnz, hipMemcpyDeviceToHost, h->stream));
        if (eps && h->nnz)
            UL_HIP(hipMemcpyAsync(eps, h->eps, sizeof(float) * h->nnz, hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipStreamSynchronize(h->stream));
        if (nnz_kept) *nnz_kept = h->nnz;
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_layout_stats(const umap_layout *h, umap_layout_stats_t *out)
{
    if (!h || !out) return fail(UMAP_E_INVAL, "handle or out is NULL");
    umap_layout_stats_t s = h->st;
    s.n = h->n;
    s.n_components = h->dim;
    s.n_epochs = h->n_epochs;
    s.neg_rate = h->neg_rate;
    s.nnz_input = h->nnz_in;
    s.nnz_kept = h->nnz;
    s.max_degree = h->max_degree;
    s.w_max = h->w_max;
    s.table_ranges = 1 << h->lg_phases;
    s.kernel = h->kernel;
    s.mode = h->mode;
    s.row_first = h->row_first;
    s.row_last = h->row_last;
    s.n_waves = h->n_waves;
    *out = s;
    return UMAP_OK;
}

int umap_layout_set_stream(umap_layout *h, void *stream)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    try {
        UL_HIP(hipStreamSynchronize(h->stream));
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
    h->stream = static_cast<hipStream_t>(stream);
    return UMAP_OK;
}

int umap_layout_set_kernel(umap_layout *h, int32_t which)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    if (which != 0 && which != 1) return fail(UMAP_E_INVAL, "kernel must be 0 or 1, got %d", which);
    h->kernel = which;
    return UMAP_OK;
}

int umap_layout_set_epoch_timing(umap_layout *h, int32_t enabled)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    h->time_epochs = enabled != 0;
    return UMAP_OK;
}

int umap_layout_epoch_ms(const umap_layout *h, float *out_ms, int32_t capacity)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    if (capacity < 0 || (capacity > 0 && !out_ms))
        return fail(UMAP_E_INVAL, "need capacity >= 0 and out_ms != NULL when capacity > 0");
    try {
        const int32_t n = h->timed < capacity ? h->timed : capacity;
        if (n > 0) UL_HIP(hipEventSynchronize(h->ep_ev[(size_t)n]));
        for (int32_t i = 0; i < n; ++i) UL_HIP(hipEventElapsedTime(&out_ms[i], h->ep_ev[(size_t)i], h->ep_ev[(size_t)i + 1]));
        return h->timed;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_layout_set_rows(umap_layout *h, int64_t row_first, int64_t row_last)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    if (row_first < 0 || row_first >= row_last || row_last > h->n)
        return fail(UMAP_E_INVAL, "need 0 <= row_first < row_last <= n (%lld), got %lld, %lld", (long long)h->n,
                    (long long)row_first, (long long)row_last);
    try {
        UL_HIP(hipSetDevice(h->device));
        // the waves of the range: the same cost rule as for the whole graph,
        // applied to the range's units
        int64_t ends[2] = {0, 0};
        UL_HIP(hipMemcpyAsync(&ends[0], h->row_ptr + row_first, sizeof(int64_t), hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipMemcpyAsync(&ends[1], h->row_ptr + row_last, sizeof(int64_t), hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipStreamSynchronize(h->stream));
        const int64_t units = ends[1] - ends[0] + (int64_t)ul::row_weight(h->dim) * (row_last - row_first);
        const int64_t cost = ul::wave_cost(units);
        int64_t waves = (units + cost - 1) / cost;
        if (waves < 1) waves = 1;
        if (waves > h->max_waves) return fail(UMAP_E_INVAL, "the range needs more waves than the handle holds");
        UL_HIP(ul::launch_partition(h->row_ptr, row_first, row_last, h->dim, cost, h->part, waves, h->head,
                                    h->stream));
        UL_HIP(hipStreamSynchronize(h->stream));
        h->n_waves = waves;
        h->row_first = row_first;
        h->row_last = row_last;
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_layout_set_mode(umap_layout *h, int32_t mode)
{
    if (!h) return fail(UMAP_E_INVAL, "handle is NULL");
    if (mode != UMAP_MODE_SYNC && mode != UMAP_MODE_ASYNC)
        return fail(UMAP_E_INVAL, "mode must be %d or %d, got %d", UMAP_MODE_SYNC, UMAP_MODE_ASYNC, mode);
    h->mode = mode;
    return UMAP_OK;
}

void umap_layout_destroy(umap_layout *h)
{
    if (!h) return;
    (void)hipSetDevice(h->device);
    h->release();
    delete h;
}

int umap_layout_debug_active(const umap_layout *h, int32_t epoch, uint8_t *out)
{
    if (!h || !out) return fail(UMAP_E_INVAL, "handle or out is NULL");
    if (epoch < 0 || epoch >= h->n_epochs) return fail(UMAP_E_INVAL, "epoch %d outside [0, %d)", epoch, h->n_epochs);
    if (h->nnz == 0) return UMAP_OK;
    uint8_t *d = nullptr;
    try {
        UL_HIP(hipSetDevice(h->device));
        UL_HIP(hipMallocAsync((void **)&d, h->nnz, h->stream));
        UL_HIP(ul::launch_debug_active(h->eps, h->nnz, epoch, d, h->stream));
        UL_HIP(hipMemcpyAsync(out, d, h->nnz, hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipFreeAsync(d, h->stream));
        d = nullptr;
        UL_HIP(hipStreamSynchronize(h->stream));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        if (d) (void)hipFreeAsync(d, h->stream);
        return hip_fail(f);
    }
}

int umap_layout_debug_negatives(const umap_layout *h, uint64_t seed, int32_t epoch, int64_t e_first, int64_t count,
                                uint32_t *out)
{
    if (!h || !out) return fail(UMAP_E_INVAL, "handle or out is NULL");
    if (e_first < 0 || count < 0 || e_first + count > h->nnz)
        return fail(UMAP_E_INVAL, "edge range [%lld, %lld) outside the %lld kept edges", (long long)e_first,
                    (long long)(e_first + count), (long long)h->nnz);
    if (count == 0 || h->neg_rate == 0) return UMAP_OK;
    uint32_t *d = nullptr;
    const size_t bytes = sizeof(uint32_t) * (size_t)count * (size_t)h->neg_rate;
    try {
        UL_HIP(hipSetDevice(h->device));
        UL_HIP(hipMallocAsync((void **)&d, bytes, h->stream));
        UL_HIP(ul::launch_debug_negatives((uint32_t)h->n_table, seed, epoch, e_first, count, h->neg_rate, d, h->stream));
        UL_HIP(hipMemcpyAsync(out, d, bytes, hipMemcpyDeviceToHost, h->stream));
        UL_HIP(hipFreeAsync(d, h->stream));
        d = nullptr;
        UL_HIP(hipStreamSynchronize(h->stream));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        if (d) (void)hipFreeAsync(d, h->stream);
        return hip_fail(f);
    }
}

int umap_fuzzy_graph_device(int64_t n, int32_t k, const int32_t *knn_ids, const float *knn_dists, int32_t *rows,
                            int32_t *cols, float *vals, void *stream)
{
    if (n < 1 || n >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "n must be in [1, 2^31)");
    if (k < 1 || k > 1024) return fail(UMAP_E_INVAL, "k must be in [1, 1024], got %d", k);
    if (2 * n * (int64_t)k >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "2 n k must be below 2^31");
    if (!knn_ids || !knn_dists || !rows || !cols || !vals) return fail(UMAP_E_INVAL, "a pointer argument is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *scratch = nullptr;
    try {
        int ndev = 0;
        if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return fail(UMAP_E_DEVICE, "no HIP device available");
        const int64_t np = ul::graph_partials(n, k);
        size_t bytes = 2 * need<double>(n) + need<double>(np + 1) + need<unsigned>(1);
        UL_HIP(hipMallocAsync(&scratch, bytes, s));
        Carver cv{static_cast<char *>(scratch)};
        double *rho = cv.take<double>(n);
        double *sigma = cv.take<double>(n);
        double *partial = cv.take<double>(np + 1);
        unsigned *flags = cv.take<unsigned>(1);
        UL_HIP(hipMemsetAsync(flags, 0, sizeof(unsigned), s));
        UL_HIP(ul::launch_fuzzy_graph(n, k, knn_ids, knn_dists, rows, cols, vals, rho, sigma, partial, np, flags, s));
        unsigned hflags = 0;
        UL_HIP(hipMemcpyAsync(&hflags, flags, sizeof hflags, hipMemcpyDeviceToHost, s));
        UL_HIP(hipFreeAsync(scratch, s));
        scratch = nullptr;
        UL_HIP(hipStreamSynchronize(s));
        if (hflags & ul::kBadIndex) return fail(UMAP_E_INVAL, "a neighbour id is outside [0, n)");
        if (hflags & ul::kBadValue) return fail(UMAP_E_INVAL, "a neighbour distance is not finite");
        return UMAP_OK;
    } catch (const HipFailure &f) {
        if (scratch) (void)hipFreeAsync(scratch, s);
        return hip_fail(f);
    }
}

}  // extern "C"

namespace {

// Scratch of umap_fuzzy_graph_device_noalloc, one copy per GPU for the life of
// the process: rho and sigma (fp64 per row), the partial sums of the mean
// distance (fp64, one per 4096 distances, plus the total) and the error flags,
// for up to kNoAllocMaxRows rows (2 n k < 2^31 bounds the partial sums).
constexpr int64_t kNoAllocMaxRows = (int64_t)1 << 20;
constexpr size_t kNoAllocBytes = 2 * (((size_t)8 << 20)) + ((((size_t)1 << 18) + 1) * 8 + 255) / 256 * 256 + 256;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

// Device address of this GPU's copy of `scratch`, looked up once per device
// with that device current (in host code the array's name is not a device
// address).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

char *noalloc_scratch()
{
    int dev = 0;
    UL_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) throw HipFailure{hipErrorInvalidDevice, "hipGetDevice (device index)"};
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        UL_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        g_scratch_ptr[dev] = p;
    }
    return static_cast<char *>(g_scratch_ptr[dev]);
}

}  // namespace

extern "C" {

int umap_fuzzy_graph_device_noalloc(int64_t n, int32_t k, const int32_t *knn_ids, const float *knn_dists,
                                    int32_t *rows, int32_t *cols, float *vals, void *stream)
{
    if (n < 1 || n > kNoAllocMaxRows)
        return fail(UMAP_E_INVAL, "n must be in [1, %lld] for the no-allocation entry point, got %lld",
                    (long long)kNoAllocMaxRows, (long long)n);
    if (k < 1 || k > 1024) return fail(UMAP_E_INVAL, "k must be in [1, 1024], got %d", k);
    if (2 * n * (int64_t)k >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "2 n k must be below 2^31");
    if (!knn_ids || !knn_dists || !rows || !cols || !vals) return fail(UMAP_E_INVAL, "a pointer argument is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    try {
        int ndev = 0;
        if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return fail(UMAP_E_DEVICE, "no HIP device available");
        const int64_t np = ul::graph_partials(n, k);
        Carver cv{noalloc_scratch()};
        double *rho = cv.take<double>(n);
        double *sigma = cv.take<double>(n);
        double *partial = cv.take<double>(np + 1);
        unsigned long long *flags = cv.take<unsigned long long>(1);
        if (cv.off > kNoAllocBytes) return fail(UMAP_E_INVAL, "scratch of %zu bytes exceeds the static %zu", cv.off,
                                                kNoAllocBytes);
        // flags start at zero (a fill kernel: no memset node if the caller captures)
        UL_HIP(ul::launch_zero_u64(flags, 1, s));
        UL_HIP(ul::launch_fuzzy_graph(n, k, knn_ids, knn_dists, rows, cols, vals, rho, sigma, partial, np,
                                      reinterpret_cast<unsigned *>(flags), s));
        unsigned long long hflags = 0;
        UL_HIP(hipMemcpyAsync(&hflags, flags, sizeof hflags, hipMemcpyDeviceToHost, s));
        UL_HIP(hipStreamSynchronize(s));
        if (hflags & ul::kBadIndex) return fail(UMAP_E_INVAL, "a neighbour id is outside [0, n)");
        if (hflags & ul::kBadValue) return fail(UMAP_E_INVAL, "a neighbour distance is not finite");
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    } catch (...) {
        return fail(UMAP_E_NOMEM, "unexpected host failure");
    }
}

int umap_trustworthiness(const float *X, int64_t n, int32_t d, const float *Y, int32_t dim, int32_t k, double *out,
                         void *stream)
{
    if (!X || !Y || !out) return fail(UMAP_E_INVAL, "X, Y and out must not be NULL");
    if (n < 1 || n >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "n must be in [1, 2^31), got %lld", (long long)n);
    if (d < 1) return fail(UMAP_E_INVAL, "d must be >= 1, got %d", d);
    if (dim < 1 || dim > 16) return fail(UMAP_E_INVAL, "dim must be in [1, 16], got %d", dim);
    if (k < 1 || k > 64) return fail(UMAP_E_INVAL, "k must be in [1, 64], got %d", k);
    if (2 * n - 3 * (int64_t)k - 1 <= 0) return fail(UMAP_E_INVAL, "need 2n - 3k - 1 > 0 (n = %lld, k = %d)", (long long)n, k);
    if (n * (int64_t)k >= ((int64_t)1 << 31)) return fail(UMAP_E_INVAL, "n k must be below 2^31");
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *scratch = nullptr;
    try {
        int ndev = 0;
        if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return fail(UMAP_E_DEVICE, "no HIP device available");
        const size_t nk = (size_t)n * (size_t)k;
        size_t bytes = need<float>(n) + need<int32_t>(nk) + need<float>(nk) + need<int32_t>(nk) + need<int64_t>(n) +
                       need<unsigned long long>(1) + need<unsigned>(1);
        UL_HIP(hipMallocAsync(&scratch, bytes, s));
        Carver cv{static_cast<char *>(scratch)};
        float *nx = cv.take<float>(n);
        int32_t *nbr = cv.take<int32_t>(nk);
        float *thr = cv.take<float>(nk);
        int32_t *cnt = cv.take<int32_t>(nk);
        int64_t *pen = cv.take<int64_t>(n);
        unsigned long long *sum = cv.take<unsigned long long>(1);
        unsigned *flags = cv.take<unsigned>(1);
        UL_HIP(hipMemsetAsync(flags, 0, sizeof(unsigned), s));
        UL_HIP(ul::launch_trustworthiness(X, n, d, Y, dim, k, nx, nbr, thr, cnt, pen, sum, flags, s));
        unsigned long long hsum = 0;
        unsigned hflags = 0;
        UL_HIP(hipMemcpyAsync(&hsum, sum, sizeof hsum, hipMemcpyDeviceToHost, s));
        UL_HIP(hipMemcpyAsync(&hflags, flags, sizeof hflags, hipMemcpyDeviceToHost, s));
        UL_HIP(hipFreeAsync(scratch, s));
        scratch = nullptr;
        UL_HIP(hipStreamSynchronize(s));
        if (hflags) return fail(UMAP_E_INVAL, "the embedding has non-finite coordinates");
        const double nn = (double)n, kk = (double)k;
        *out = 1.0 - 2.0 / (nn * kk * (2.0 * nn - 3.0 * kk - 1.0)) * (double)hsum;
        return UMAP_OK;
    } catch (const HipFailure &f) {
        if (scratch) (void)hipFreeAsync(scratch, s);
        return hip_fail(f);
    }
}

int umap_probe_copy(const void *src, void *dst, int64_t bytes, void *stream)
{
    if (!src || !dst || bytes < 0 || bytes % 16) return fail(UMAP_E_INVAL, "need non-NULL pointers and bytes %% 16 == 0");
    try {
        UL_HIP(ul::launch_probe_copy(src, dst, bytes, static_cast<hipStream_t>(stream)));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

int umap_probe_gather(const void *table, int64_t entries, int64_t threads, int32_t iters, void *out, void *stream)
{
    if (!table || !out) return fail(UMAP_E_INVAL, "table and out must not be NULL");
    if (entries < 1 || entries > ((int64_t)1 << 32) || (entries & (entries - 1)))
        return fail(UMAP_E_INVAL, "entries must be a power of two in [1, 2^32]");
    if (threads < 256 || threads % 256 || threads / 256 > 0x7FFFFFFF)
        return fail(UMAP_E_INVAL, "threads must be a positive multiple of 256");
    if (iters < 1) return fail(UMAP_E_INVAL, "iters must be >= 1");
    try {
        UL_HIP(ul::launch_probe_gather(table, entries, threads, iters, out, static_cast<hipStream_t>(stream)));
        return UMAP_OK;
    } catch (const HipFailure &f) {
        return hip_fail(f);
    }
}

}  // extern "C"
