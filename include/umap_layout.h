/*
 * umap_layout.h -- C ABI of the MI355X (gfx950) layout-optimisation SGD of
 * GPU UMAP (Nolet et al., "Bringing UMAP Closer to the Speed of Light with
 * GPU Acceleration", AAAI 2021).
 *
 * What is computed.  Given the fuzzy union B (Eq. 2) of the neighbourhood
 * graph as a symmetric weighted COO list, the library lays out n points in
 * n_components dimensions by stochastic gradient descent on the cross-entropy
 * objective of the UMAP section: every sampled edge (i, j) of B pulls both
 * endpoints together (gradient of log Phi, Phi = 1/(1 + a d^(2b))), and each
 * sampled edge draws neg_rate vertices uniformly at random that push the
 * source away (gradient of log(1 - Phi)); embedding-updates section.  Edge e
 * of weight w_e is sampled once every eps_e = w_max / w_e epochs.  Gradient
 * components are clipped to [-4, 4]; the step size decays linearly,
 * alpha_n = 1 - n / n_epochs.  By default updates are epoch-synchronous:
 * every read of epoch n sees the layout at the start of the epoch and all
 * updates are applied at its end, which makes the result a deterministic
 * function of the seed (the exactly-repeatable mode of the reproducibility
 * section).  umap_layout_set_mode selects the asynchronous (Hogwild) mode
 * instead, the paper's default: updates land in place while the epoch runs.
 *
 * Conventions.
 *   - Every function returns UMAP_OK (0) or a negative UMAP_E_* code and, on
 *     failure, sets a thread-local message readable with
 *     umap_layout_last_error().  No C++ exception crosses the ABI.
 *   - Out-parameters are left untouched on failure.
 *   - Argument checks that need no GPU run before any HIP call.
 *   - A handle belongs to the HIP device that was current at creation and is
 *     used by one host thread at a time.  Work is enqueued on the handle's
 *     stream (the null stream unless set); calls documented as blocking
 *     synchronise that stream before returning.
 *   - Layouts are row-major: element (i, d) of an n x n_components array is
 *     at index i * n_components + d.  All embedding values are fp32.
 */
#ifndef UMAP_LAYOUT_H
#define UMAP_LAYOUT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define UMAP_OK 0
#define UMAP_E_INVAL (-1)      /* an argument or the graph is invalid          */
#define UMAP_E_ASYMMETRIC (-2) /* the kept graph is not symmetric              */
#define UMAP_E_NOMEM (-3)      /* device or host allocation failed             */
#define UMAP_E_DEVICE (-4)     /* no usable GPU, or a HIP call failed          */
#define UMAP_E_STATE (-5)      /* call not valid in the handle's current state */

#define UMAP_MODE_SYNC 0       /* epoch-synchronous updates (default)          */
#define UMAP_MODE_ASYNC 1      /* asynchronous in-place updates (Hogwild)      */

typedef struct umap_layout umap_layout;

typedef struct {
    int64_t n;              /* vertices                                          */
    int32_t n_components;   /* embedding dimension                               */
    int32_t n_epochs;       /* N                                                 */
    int32_t neg_rate;       /* negative samples per sampled edge                 */
    int32_t epochs_done;    /* epochs run by the last run / run_epochs call      */
    int64_t nnz_input;      /* entries passed to create                          */
    int64_t nnz_kept;       /* edges kept after drop and prune                   */
    int32_t max_degree;     /* largest kept row                                  */
    float w_max;            /* largest kept weight                               */
    int64_t active_edges;   /* sampled edges over the last call's epochs         */
    int64_t edge_updates;   /* active_edges * (1 + neg_rate): positive samples
                               plus drawn negatives (self draws included)        */
    double prep_ms;         /* device time of the ingest inside create           */
    double init_ms;         /* device time of the random initialisation (run)    */
    double epochs_ms;       /* device time of the last call's epoch launches     */
    int32_t table_ranges;   /* P: an epoch is one draw launch and, for P > 1,
                               P repulsion launches, each gathering from 1/P of
                               the table (with P = 1 the draw launch applies
                               the negative samples itself)                     */
    int32_t kernel;         /* epoch kernel in use (see umap_layout_set_kernel)  */
    int32_t overflow_redone; /* 1 when the last call's epochs were redone by the
                               one-thread-per-vertex kernel because a negative
                               sample found its record slot full (the result is
                               the same bit for bit; only the time is lost)    */
    int32_t mode;           /* UMAP_MODE_SYNC or UMAP_MODE_ASYNC                 */
    int64_t row_first;      /* rows the epochs update: [row_first, row_last)     */
    int64_t row_last;       /*   (umap_layout_set_rows; 0 and n by default)      */
    int64_t n_waves;        /* waves of an edge-parallel epoch launch            */
} umap_layout_stats_t;

/*
 * umap_layout_create -- ingest a host COO graph (sparse-data handling section:
 * the COO list is sorted by row with a CSR index into it).
 *
 *   out           receives the handle (NULL on failure).
 *   n             vertices, 1 <= n < 2^31.
 *   n_components  embedding dimension, 1..16.
 *   rows, cols    nnz int32 vertex ids in [0, n) (host memory, read only).
 *   vals          nnz fp32 weights of B, finite (host memory, read only).
 *   nnz           entries, 0 <= nnz < 2^31; nnz = 0 gives a graph without
 *                 edges (a run only initialises the layout).
 *   a, b          Phi(d) = 1 / (1 + a d^(2b)) (Eq. 3's smooth form), > 0.
 *   n_epochs      1 <= N < 2^24.
 *   neg_rate      negative samples per sampled edge, 0 <= R < 2^16.
 *
 * The inputs are copied; the caller keeps ownership.  On the device the
 * ingest drops entries with val <= 0 and self loops, takes w_max = the largest
 * remaining value, prunes entries with val < w_max / N (fp32), sorts the rest
 * by (row, col) -- edge e is the position in that order -- and stores
 * eps_e = w_max / val_e (fp32).  The kept graph must be symmetric: every
 * kept (i, j, v) needs a kept (j, i) with bit-equal v.
 * Errors: UMAP_E_INVAL (a scalar out of range, an index outside [0, n), a
 * non-finite value, a kept (i, j) listed twice, a row too long for the
 * accumulator), UMAP_E_ASYMMETRIC, UMAP_E_NOMEM, UMAP_E_DEVICE.  Blocking.
 */
int umap_layout_create(umap_layout **out, int64_t n, int32_t n_components, const int32_t *rows,
                       const int32_t *cols, const float *vals, int64_t nnz, float a, float b,
                       int32_t n_epochs, int32_t neg_rate);

/*
 * umap_layout_create_device -- as umap_layout_create, with rows, cols and
 * vals in device memory of the current device (read only; the caller keeps
 * ownership and may free them once the call returns).  `stream` (a
 * hipStream_t, or NULL for the null stream) becomes the handle's stream.
 * Index and value checks run on the device.  Blocking.
 */
int umap_layout_create_device(umap_layout **out, int64_t n, int32_t n_components, const int32_t *rows,
                              const int32_t *cols, const float *vals, int64_t nnz, float a, float b,
                              int32_t n_epochs, int32_t neg_rate, void *stream);

/*
 * umap_layout_run -- random initial layout, uniform on [-10, 10) per
 * coordinate from the seed (embedding-updates section: random
 * initialisation), then epochs 0 .. N-1.  Same seed, same graph: bit-identical
 * output in the synchronous mode (UMAP_MODE_SYNC).  Blocking.
 */
int umap_layout_run(umap_layout *h, uint64_t seed);

/*
 * umap_layout_init -- only the initialisation of umap_layout_run: the uniform
 * random layout on [-10, 10) from `seed` for a fit (embedding-updates section),
 * the weighted mean of the kept neighbours for a transform.  Afterwards
 * umap_layout_run_epochs(h, seed, 0, N) equals umap_layout_run(h, seed), and
 * the epochs can be taken in pieces (e.g. to look at the layout in between).
 * Blocking.
 */
int umap_layout_init(umap_layout *h, uint64_t seed);

/*
 * umap_layout_run_epochs -- epochs first .. last-1 (0 <= first <= last <= N)
 * from the current layout, without initialisation.  Because the random
 * streams are counter-based, running 0..m then m..N equals one run of 0..N.
 * UMAP_E_STATE if no layout is present (no run and no set_embedding yet).
 * Blocking.
 */
int umap_layout_run_epochs(umap_layout *h, uint64_t seed, int32_t first, int32_t last);

/* umap_layout_get -- copy the n x n_components fp32 layout into host memory
 * owned by the caller.  UMAP_E_STATE before the first run / set_embedding.
 * Blocking. */
int umap_layout_get(const umap_layout *h, float *out);

/* umap_layout_get_device -- copy the layout into device memory `dev_out`
 * (n x n_components fp32, caller-owned) on the handle's stream; not blocking.
 * UMAP_E_STATE before the first run / set_embedding. */
int umap_layout_get_device(const umap_layout *h, float *dev_out);

/* umap_layout_set_embedding -- replace the layout with n x n_components fp32
 * values from host memory (read only).  Blocking. */
int umap_layout_set_embedding(umap_layout *h, const float *host);

/* umap_layout_get_graph -- copy the kept graph to host memory: row_ptr
 * (n + 1 int64), col (nnz_kept int32), eps (nnz_kept fp32).  Any array
 * pointer may be NULL to skip it; nnz_kept may be NULL.  Blocking. */
int umap_layout_get_graph(const umap_layout *h, int64_t *row_ptr, int32_t *col, float *eps,
                          int64_t *nnz_kept);

/* umap_layout_stats -- counters and device timings of the handle. */
int umap_layout_stats(const umap_layout *h, umap_layout_stats_t *out);

/* umap_layout_set_epoch_timing -- enabled != 0: later run / run_epochs calls
 * record a HIP event on the handle's stream before each of their first
 * UMAP_MAX_TIMED_EPOCHS epochs and one after the last of them (the events are
 * created on first use and kept until destroy); 0 turns it off.  Off by
 * default: an event per epoch costs a few microseconds of launch time. */
#define UMAP_MAX_TIMED_EPOCHS 4096
int umap_layout_set_epoch_timing(umap_layout *h, int32_t enabled);

/* umap_layout_epoch_ms -- device time of each timed epoch of the last call
 * (the time between the events around it, on the handle's stream), in ms, into
 * out_ms[0 .. min(count, capacity)); returns count >= 0, the epochs the last
 * call timed (0 when timing was off), or a negative UMAP_E_* code (NULL
 * handle or out_ms with capacity > 0, capacity < 0).  If the last call's
 * epochs were redone (stats.overflow_redone), these are the redo's times.
 * Blocking. */
int umap_layout_epoch_ms(const umap_layout *h, float *out_ms, int32_t capacity);

/* umap_layout_set_stream -- enqueue later work on `stream` (hipStream_t or
 * NULL).  The caller keeps ownership of the stream and must keep it alive
 * while the handle uses it. */
int umap_layout_set_stream(umap_layout *h, void *stream);

/* umap_layout_destroy -- free all device memory of the handle (waits for its
 * stream).  NULL is a no-op. */
void umap_layout_destroy(umap_layout *h);

/* umap_layout_last_error -- message of the last failing call on this thread
 * ("" if none).  Valid until the next failing call on this thread. */
const char *umap_layout_last_error(void);

/*
 * umap_transform_create -- a handle that lays out n_new new points against a
 * frozen trained layout (inference: the model section keeps the training kNN
 * index to map new points; the embedding-updates section moves only the new
 * points).  The graph is bipartite: row i is new point i, column j is row j of
 * the table, with weight v (e.g. the membership strength of Eq. 1 of the new
 * point's kNN among the training points; no union, no symmetry).
 *
 *   out        receives the handle (NULL on failure).
 *   n_new      new points, 1 <= n_new < 2^31.
 *   n_components  embedding dimension, 1..16 (the table's).
 *   table      n_table x n_components fp32 trained layout, row-major, host
 *              memory (read only; copied, the caller keeps ownership).
 *   n_table    rows of the table, 1 <= n_table < 2^31.
 *   rows, cols nnz int32 indices, rows in [0, n_new), cols in [0, n_table)
 *              (host memory, read only).  Equal row and column indices are
 *              ordinary edges here.
 *   vals       nnz fp32 weights, finite; entries <= 0 are dropped, the rest
 *              pruned below w_max / n_epochs as in a fit.
 *   a, b, n_epochs, neg_rate  as for umap_layout_create (negative samples are
 *              drawn from the table's rows).
 *
 * The handle takes the same calls as a fit's, with these differences:
 * umap_layout_run initialises every new point at the mean of its kept
 * neighbours' table rows weighted by 1/eps_e (the origin when it has none) --
 * the seed then only keys the negative samples -- and each sampled edge (i, j)
 * moves new point i by alpha_n x the clipped attraction toward table row j
 * (once: the table does not move and there is no reverse edge), each negative
 * sample k by alpha_n x the clipped repulsion from table row k.  Updates are
 * epoch-synchronous and deterministic; UMAP_MODE_ASYNC is not available
 * (UMAP_E_INVAL from the run).  Errors: UMAP_E_INVAL for bad arguments or
 * indices, UMAP_E_NOMEM, UMAP_E_DEVICE; never UMAP_E_ASYMMETRIC.
 */
int umap_transform_create(umap_layout **out, int64_t n_new, int32_t n_components, const float *table,
                          int64_t n_table, const int32_t *rows, const int32_t *cols, const float *vals, int64_t nnz,
                          float a, float b, int32_t n_epochs, int32_t neg_rate);

/* ---- diagnostics (tests, measurement) ---------------------------------- */

/* umap_layout_debug_active -- host array of nnz_kept bytes: 1 where edge e is
 * sampled in `epoch` (floor((epoch + 1) / eps_e) > floor(epoch / eps_e),
 * fp32), computed on the device.  Blocking. */
int umap_layout_debug_active(const umap_layout *h, int32_t epoch, uint8_t *out);

/* umap_layout_debug_negatives -- host array of count x neg_rate uint32: the
 * negative-sample vertices the epoch kernel draws for edges
 * e_first .. e_first + count - 1 in `epoch` with `seed` (vertices of the
 * table for a transform handle), computed on the device by the same routine.  0 <= e_first, e_first + count <= nnz_kept.  Blocking. */
int umap_layout_debug_negatives(const umap_layout *h, uint64_t seed, int32_t epoch, int64_t e_first,
                                int64_t count, uint32_t *out);

/* umap_layout_set_kernel -- choose the epoch kernel: 0 = edge-parallel
 * wavefront kernel (default), 1 = one thread per vertex.  Both compute the
 * same result bit for bit.  In UMAP_MODE_ASYNC: 0 = range-ordered, 1 =
 * per-edge (see umap_layout_set_mode). */
int umap_layout_set_kernel(umap_layout *h, int32_t which);

/* umap_layout_set_mode -- how later runs apply their updates (embedding-updates
 * and reproducibility sections):
 *   UMAP_MODE_SYNC   epoch-synchronous (default): E_{n+1} = E_n + alpha_n x
 *                    the sum of the epoch's terms, every term computed from
 *                    E_n; deterministic, bit-identical for both kernels.
 *   UMAP_MODE_ASYNC  asynchronous, in place (Hogwild): updates land in the
 *                    layout while the epoch runs and reads see whatever has
 *                    been written, so the result depends on the timing of
 *                    the GPU's threads and is not repeatable bit for bit.
 *                    Same schedule, negative draws, clip and step size as
 *                    the synchronous mode.  Two kernels (set_kernel):
 *                    0 (default) range-ordered: the launches of a
 *                      synchronous epoch (sampled edges with their
 *                      attractions, then the negative samples of each table
 *                      range) each add alpha_n x their sums to the rows they
 *                      own as they finish;
 *                    1 per-edge: one thread per sampled edge applies
 *                      alpha_n x the clipped attraction to its source (a
 *                      private copy) and the opposite change to its
 *                      destination, then each negative sample's repulsion to
 *                      the private copy in turn, and adds the source's
 *                      change to the layout; needs rows of fewer than
 *                      2^24 - 8192 edges (UMAP_E_INVAL from the run
 *                      otherwise).
 * Any other value is UMAP_E_INVAL.  Takes effect at the next run. */
int umap_layout_set_mode(umap_layout *h, int32_t mode);

/* umap_layout_set_rows -- later epochs update only the rows [row_first,
 * row_last): one GPU's share of a layout sharded by contiguous row ranges.
 * The epoch of the embedding-updates section (epoch-synchronous reading) is a
 * sum of terms per row, each read from the snapshot E_n; a GPU that owns a
 * range computes its rows' sums from a full replica of E_n, and an
 * all-gather of the rows would end the epoch.  Here the rows outside the
 * range keep their values (they stand for the rows other GPUs own).  The
 * negative samples are still drawn from all vertices and keyed by the global
 * edge ids, and the sums are exact, so each row of the range is bit-identical
 * to the same row of an epoch over all rows from the same layout.  The waves
 * of the edge-parallel kernel are re-cut for the range (the same cost rule
 * applied to its edges and rows); init still sets every row.  Synchronous
 * mode only (a run in UMAP_MODE_ASYNC with a range is UMAP_E_INVAL).
 * umap_layout_set_rows(h, 0, n) restores the default.  Errors: UMAP_E_INVAL
 * unless 0 <= row_first < row_last <= n; UMAP_E_DEVICE.  Blocking. */
int umap_layout_set_rows(umap_layout *h, int64_t row_first, int64_t row_last);

/* ---- quality ------------------------------------------------------------- */

/*
 * umap_trustworthiness -- T(k) of an embedding on the GPU (the batched pairwise
 * distance computation of Alg. 1, with the normalisation of Venna and Kaski's
 * definition that the experiments section cites):
 *   T(k) = 1 - 2 / (n k (2n - 3k - 1)) sum_i sum_{j in N^_k(i)} max(0, r(i, j) - k),
 * N^_k(i) the k nearest neighbours of i in the embedding (ties by index),
 * r(i, j) the 1-based rank of j by input distance from i (self excluded, ties by
 * index).
 *   X    n x d fp32 input points, row-major, device memory (read only).
 *   Y    n x dim fp32 embedding, row-major, device memory (read only), dim 1..16.
 *   k    1..64, with 2n - 3k - 1 > 0 and n k < 2^31.
 *   out  host double, receives T.
 * Distances are fp32 (input distances as |x_i|^2 + |x_j|^2 - 2 x_i . x_j with
 * the dot products on the matrix cores): a pair closer to a tie than fp32
 * resolves can rank differently from an exact evaluation, each such pair
 * moving T by about 1 / (n^2 k).  Errors: UMAP_E_INVAL (arguments, a non-finite
 * embedding), UMAP_E_NOMEM, UMAP_E_DEVICE.  Scratch of about 8 n k bytes is
 * allocated on `stream` (NULL: null stream) and freed.  Blocking.
 */
int umap_trustworthiness(const float *X, int64_t n, int32_t d, const float *Y, int32_t dim, int32_t k, double *out,
                         void *stream);

/* ---- input side --------------------------------------------------------- */

/*
 * umap_fuzzy_graph_device -- from a kNN graph (n x k neighbour ids and
 * distances, row-major, device memory; neighbourhood-weighting section) build
 * B on the device: rho_i (the smallest positive distance of row i), sigma_i
 * (bisection so that sum_j exp(-max(0, d_ij - rho_i)/sigma_i) = log2 k, Eq. 1,
 * floored at 1e-3 of the row's mean distance), A_ij, and the t-conorm
 * A + A^T - A o A^T (Eq. 2), in fp64, rounded to fp32.
 * Output: 2 n k COO slots in caller-owned device memory (rows, cols int32;
 * vals fp32).  Slot i*k+s holds (i, j, B_ij) for j = ids[i*k+s]; slot
 * n*k + i*k + s holds (j, i, B_ij) when i is not among j's neighbours and a
 * placeholder of value 0 otherwise (placeholders and self entries are dropped
 * by create).  Errors: UMAP_E_INVAL (n < 1, k < 1, k > 1024, 2nk >= 2^31, an
 * id outside [0, n), a non-finite distance).  Blocking.
 */
int umap_fuzzy_graph_device(int64_t n, int32_t k, const int32_t *knn_ids, const float *knn_dists,
                            int32_t *rows, int32_t *cols, float *vals, void *stream);

/*
 * umap_fuzzy_graph_device_noalloc -- umap_fuzzy_graph_device for callers that
 * cannot allocate device memory (code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid hipMalloc): the same kernels and the
 * same result bit for bit, with its scratch (rho, sigma, the partial sums of
 * the mean distance, the error flags: about 16 n bytes + 2 MB) taken from a
 * static array that the library keeps on each GPU it runs on until the process
 * ends (about 18 MB per GPU).  It calls no hipMalloc, hipFree or allocating
 * library routine.  Arguments, layout and errors as umap_fuzzy_graph_device,
 * and n <= 1,048,576 (UMAP_E_INVAL beyond).  Every call on one GPU uses that
 * GPU's one array: calls that overlap on a GPU (other host threads, other
 * streams) race and must be serialised by the caller.  Blocking.
 */
int umap_fuzzy_graph_device_noalloc(int64_t n, int32_t k, const int32_t *knn_ids, const float *knn_dists,
                                    int32_t *rows, int32_t *cols, float *vals, void *stream);

/* umap_fit_ab -- least-squares (a, b) of 1/(1 + a x^(2b)) against Eq. 3's
 * target (1 below min_dist, exp(-(x - min_dist)/spread) above) on 300 points
 * of [0, 3 spread].  spread > 0, 0 <= min_dist < 3 spread.  Host only. */
int umap_fit_ab(float spread, float min_dist, float *a, float *b);

/* ---- roofline probes ---------------------------------------------------- */

/* umap_probe_copy -- stream `bytes` (a multiple of 16) from src to dst on
 * `stream` with 16-byte vector loads and stores; not blocking. */
int umap_probe_copy(const void *src, void *dst, int64_t bytes, void *stream);

/* umap_probe_gather -- random 8-byte gathers: each of `threads` threads (a
 * positive multiple of 256) reads iters x 16 entries at hashed positions of
 * `table`, `entries` (a power of two) pairs of fp32 in device memory, the
 * access pattern of the negative-sample repulsions without their arithmetic.
 * `out` is device memory for `threads` fp32 (written only so the loads are not
 * optimised away).  Measures the cache-served gather ceiling of a table of a
 * given size.  On `stream`; not blocking. */
int umap_probe_gather(const void *table, int64_t entries, int64_t threads, int32_t iters, void *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* UMAP_LAYOUT_H */
