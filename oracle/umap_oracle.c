/*
 * umap_oracle.c -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * A plain, slow, obviously-correct CPU reference for the layout path of GPU UMAP
 * (Nolet et al., "Bringing UMAP Closer to the Speed of Light with GPU
 * Acceleration", AAAI 2021).  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, constant table or helper with the GPU library; the two agree only
 * through the documented readings of the paper.
 *
 * State and arithmetic are fp64.  The edge schedule (prune threshold, epochs
 * per sample, the per-epoch predicate) is evaluated in fp32 IEEE, because it
 * turns floating point into integer decisions that both sides must take in the
 * same precision.  Random numbers come from Philox4x32-10 as defined by Salmon,
 * Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11).
 *
 * Where the paper is silent or garbled (smooth-kNN constants, the union's
 * sign, the schedule, constants gamma = 1, eps = 1e-3, clip 4, the RNG counter
 * layout) each function states the reading it takes beside its code; the GPU
 * library takes the same readings.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (SC'11, section 3: Philox with N = 4, W = 32, 10 rounds).   */
/* ------------------------------------------------------------------------ */

/* Multipliers and Weyl key increments given for Philox4x32 in SC'11. */
static const uint32_t PH_MUL_A = 0xD2511F53u;
static const uint32_t PH_MUL_B = 0xCD9E8D57u;
static const uint32_t PH_KEY_A = 0x9E3779B9u; /* golden ratio */
static const uint32_t PH_KEY_B = 0xBB67AE85u; /* sqrt(3) - 1 */

/* One Philox round: two 32x32->64 products; the high halves are xored with the
 * other two counter words and the round key, then the words are permuted. */
static void philox_round(uint32_t x[4], uint32_t k0, uint32_t k1)
{
    uint64_t pa = (uint64_t)PH_MUL_A * (uint64_t)x[0];
    uint64_t pb = (uint64_t)PH_MUL_B * (uint64_t)x[2];
    uint32_t y0 = (uint32_t)(pb >> 32) ^ x[1] ^ k0;
    uint32_t y1 = (uint32_t)pb;
    uint32_t y2 = (uint32_t)(pa >> 32) ^ x[3] ^ k1;
    uint32_t y3 = (uint32_t)pa;
    x[0] = y0; x[1] = y1; x[2] = y2; x[3] = y3;
}

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += PH_KEY_A; k1 += PH_KEY_B; }
        philox_round(x, k0, k1);
    }
    out[0] = x[0]; out[1] = x[1]; out[2] = x[2]; out[3] = x[3];
}

/* Batch form for tests: count counters (4 words each) -> 4 words each. */
void orc_philox_batch(const uint32_t key[2], int64_t count, const uint32_t *ctrs, uint32_t *out)
{
    for (int64_t t = 0; t < count; ++t) orc_philox4x32_10(ctrs + 4 * t, key, out + 4 * t);
}

/* Stream layout (a reading: the paper only says a seed controls the random
 * state).  Key = (low, high) 32-bit halves of the seed.
 *   init:     counter (lo32 i, hi32 i, d / 4, TAG_INIT),       word d % 4
 *   negative: counter (lo32 e, hi32 e, epoch, TAG_NEG | r / 4), word r % 4   */
#define ORC_TAG_INIT 0x494E0000u
#define ORC_TAG_NEG  0x4E470000u

static uint32_t stream_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, int w)
{
    uint32_t ctr[4] = {c0, c1, c2, c3};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    orc_philox4x32_10(ctr, key, out);
    return out[w];
}

/* Negative sample r of edge e in epoch `epoch`: a vertex drawn uniformly from
 * 0..n-1 by the multiply-high map of one 32-bit word. */
uint32_t orc_negative_vertex(uint64_t seed, int64_t e, int32_t epoch, int32_t r, int64_t n)
{
    uint32_t u = stream_word(seed, (uint32_t)(uint64_t)e, (uint32_t)((uint64_t)e >> 32),
                             (uint32_t)epoch, ORC_TAG_NEG | (uint32_t)(r >> 2), r & 3);
    return (uint32_t)(((uint64_t)u * (uint64_t)n) >> 32);
}

void orc_negative_batch(uint64_t seed, int32_t epoch, int64_t e_first, int64_t count,
                        int32_t neg_rate, int64_t n, uint32_t *out)
{
    for (int64_t t = 0; t < count; ++t)
        for (int32_t r = 0; r < neg_rate; ++r)
            out[t * neg_rate + r] = orc_negative_vertex(seed, e_first + t, epoch, r, n);
}

/* Random initial layout: uniform on [-10, 10) per coordinate (the paper's
 * random initialisation; its range is the workload's).  The top 24 bits of the
 * word give an exact value in [-1, 1), scaled once by 10 in fp32. */
void orc_init(int64_t n, int32_t dim, uint64_t seed, float *out)
{
    for (int64_t i = 0; i < n; ++i)
        for (int32_t d = 0; d < dim; ++d) {
            uint32_t u = stream_word(seed, (uint32_t)(uint64_t)i, (uint32_t)((uint64_t)i >> 32),
                                     (uint32_t)(d >> 2), ORC_TAG_INIT, d & 3);
            float unit = (float)((int32_t)(u >> 8) - (1 << 23)) * 0x1p-23f;
            out[i * dim + d] = unit * 10.0f;
        }
}

/* ------------------------------------------------------------------------ */
/* Neighbourhood weighting (Eq. 1) and the fuzzy union (Eq. 2).              */
/* ------------------------------------------------------------------------ */

/* rho_i: distance to the closest neighbour at non-zero distance (0 if none).
 * sigma_i: the normaliser for which sum_j exp(-max(0, d_ij - rho_i)/sigma_i)
 * equals log2(k), found by bisection (start 1, doubling while unbounded,
 * at most 64 steps, stop when within 1e-5), floored at 1e-3 times the mean
 * neighbour distance of the row (the global mean if rho_i is 0). */
void orc_smooth_knn(int64_t n, int32_t k, const float *dists, double *rho, double *sigma)
{
    const double target = log2((double)k);
    double gsum = 0.0;
    for (int64_t t = 0; t < n * (int64_t)k; ++t) gsum += (double)dists[t];
    const double gmean = n > 0 ? gsum / ((double)n * (double)k) : 0.0;

#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const float *d = dists + i * k;
        double r = 0.0;
        int found = 0;
        double rsum = 0.0;
        for (int32_t j = 0; j < k; ++j) {
            double dj = (double)d[j];
            rsum += dj;
            if (dj > 0.0 && (!found || dj < r)) { r = dj; found = 1; }
        }
        double lo = 0.0, hi = INFINITY, s = 1.0;
        for (int it = 0; it < 64; ++it) {
            double f = 0.0;
            for (int32_t j = 0; j < k; ++j) {
                double x = (double)d[j] - r;
                f += x > 0.0 ? exp(-x / s) : 1.0;
            }
            if (fabs(f - target) < 1e-5) break;
            if (f > target) hi = s; else lo = s;
            s = isinf(hi) ? 2.0 * s : 0.5 * (lo + hi);
        }
        double fl = r > 0.0 ? 1e-3 * (rsum / (double)k) : 1e-3 * gmean;
        if (s < fl) s = fl;
        rho[i] = r;
        sigma[i] = s;
    }
}

/* Membership strength of each directed kNN edge (the summand of Eq. 1). */
void orc_membership(int64_t n, int32_t k, const float *dists, const double *rho, const double *sigma,
                    double *A)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        for (int32_t j = 0; j < k; ++j) {
            double x = (double)dists[i * k + j] - rho[i];
            A[i * k + j] = exp(-(x > 0.0 ? x : 0.0) / sigma[i]);
        }
}

/* Fuzzy union B = A + A^T - A o A^T (the probabilistic t-conorm applied
 * elementwise over the union of both structures).  Input: the n x k id and
 * membership arrays of the directed kNN graph.  Output: B as COO sorted by
 * (row, col), capacity 2*n*k, fp64 values.  Self entries are dropped.
 * Returns the entry count, or -1 if a row lists a neighbour twice or an id is
 * out of range. */
int64_t orc_fuzzy_union(int64_t n, int32_t k, const int32_t *ids, const double *A,
                        int32_t *rows, int32_t *cols, double *vals)
{
    /* value of the directed edge (i -> j), or 0 when j is not a neighbour of i */
    int64_t m = 0;
    int64_t *cnt = calloc((size_t)n + 1, sizeof(int64_t));
    if (!cnt) return -1;
    for (int64_t i = 0; i < n; ++i)
        for (int32_t a = 0; a < k; ++a) {
            int32_t j = ids[i * k + a];
            if (j < 0 || j >= n) { free(cnt); return -1; }
            for (int32_t b2 = 0; b2 < a; ++b2)
                if (ids[i * k + b2] == j) { free(cnt); return -1; }
        }
    /* emit both orientations of every pair once: (i, j) from i's list, and
     * (j, i) from i's list only when i is not in j's list */
    int32_t *tr = malloc(sizeof(int32_t) * 2 * (size_t)n * (size_t)k);
    int32_t *tc = malloc(sizeof(int32_t) * 2 * (size_t)n * (size_t)k);
    double *tv = malloc(sizeof(double) * 2 * (size_t)n * (size_t)k);
    if (!tr || !tc || !tv) { free(cnt); free(tr); free(tc); free(tv); return -1; }
    for (int64_t i = 0; i < n; ++i)
        for (int32_t a = 0; a < k; ++a) {
            int32_t j = ids[i * k + a];
            if (j == i) continue;
            double aij = A[i * k + a];
            double aji = 0.0;
            int mutual = 0;
            for (int32_t b2 = 0; b2 < k; ++b2)
                if (ids[(int64_t)j * k + b2] == (int32_t)i) { aji = A[(int64_t)j * k + b2]; mutual = 1; }
            double bij = aij + aji - aij * aji;
            tr[m] = (int32_t)i; tc[m] = j; tv[m] = bij; ++m;
            if (!mutual) { tr[m] = j; tc[m] = (int32_t)i; tv[m] = bij; ++m; }
        }
    /* counting sort by row, then insertion sort by column inside each row */
    for (int64_t t = 0; t < m; ++t) cnt[tr[t] + 1]++;
    for (int64_t i = 0; i < n; ++i) cnt[i + 1] += cnt[i];
    int64_t *pos = malloc(sizeof(int64_t) * ((size_t)n + 1));
    memcpy(pos, cnt, sizeof(int64_t) * ((size_t)n + 1));
    for (int64_t t = 0; t < m; ++t) {
        int64_t p = pos[tr[t]]++;
        rows[p] = tr[t]; cols[p] = tc[t]; vals[p] = tv[t];
    }
    for (int64_t i = 0; i < n; ++i)
        for (int64_t p = cnt[i] + 1; p < cnt[i + 1]; ++p) {
            int32_t c = cols[p];
            double v = vals[p];
            int64_t q = p - 1;
            while (q >= cnt[i] && cols[q] > c) { cols[q + 1] = cols[q]; vals[q + 1] = vals[q]; --q; }
            cols[q + 1] = c; vals[q + 1] = v;
        }
    free(pos); free(cnt); free(tr); free(tc); free(tv);
    return m;
}

/* ------------------------------------------------------------------------ */
/* Fit of the smooth curve 1 / (1 + a x^(2b)) to the target of Eq. 3.        */
/* ------------------------------------------------------------------------ */

/* Target: 1 for x < min_dist, exp(-(x - min_dist)/spread) beyond; 300 points
 * on [0, 3 spread]; Levenberg-Marquardt least squares from (a, b) = (1, 1). */
static double ab_cost(double a, double b, const double *x, const double *y, int m)
{
    double c = 0.0;
    for (int t = 0; t < m; ++t) {
        double p = x[t] > 0.0 ? 1.0 / (1.0 + a * pow(x[t], 2.0 * b)) : 1.0;
        c += (p - y[t]) * (p - y[t]);
    }
    return c;
}

int orc_fit_ab(double spread, double min_dist, double *a_out, double *b_out)
{
    enum { M = 300 };
    double x[M], y[M];
    for (int t = 0; t < M; ++t) {
        x[t] = 3.0 * spread * (double)t / (double)(M - 1);
        y[t] = x[t] < min_dist ? 1.0 : exp(-(x[t] - min_dist) / spread);
    }
    double a = 1.0, b = 1.0, lam = 1e-3;
    double cost = ab_cost(a, b, x, y, M);
    for (int it = 0; it < 1000; ++it) {
        /* normal equations J^T J and J^T r of the residual r = p - y */
        double jaa = 0, jab = 0, jbb = 0, ga = 0, gb = 0;
        for (int t = 0; t < M; ++t) {
            if (x[t] <= 0.0) continue; /* p = 1 and both derivatives vanish at x = 0 */
            double xb = pow(x[t], 2.0 * b);
            double den = 1.0 + a * xb;
            double p = 1.0 / den;
            double dpa = -xb / (den * den);
            double dpb = -a * xb * 2.0 * log(x[t]) / (den * den);
            double r = p - y[t];
            jaa += dpa * dpa; jab += dpa * dpb; jbb += dpb * dpb;
            ga += dpa * r; gb += dpb * r;
        }
        int accepted = 0;
        for (int tries = 0; tries < 50 && !accepted; ++tries) {
            double maa = jaa * (1.0 + lam), mbb = jbb * (1.0 + lam);
            double det = maa * mbb - jab * jab;
            double da = -(mbb * ga - jab * gb) / det;
            double db = -(maa * gb - jab * ga) / det;
            double nc = ab_cost(a + da, b + db, x, y, M);
            if (nc < cost) {
                double rel = (cost - nc) / (cost > 0 ? cost : 1.0);
                a += da; b += db; cost = nc; lam *= 0.1; accepted = 1;
                if (rel < 1e-15 && fabs(da) < 1e-13 && fabs(db) < 1e-13) it = 1000;
            } else {
                lam *= 10.0;
            }
        }
        if (!accepted) break;
    }
    *a_out = a;
    *b_out = b;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Edge schedule: prune, sort by (head, tail), epochs per sample, predicate. */
/* ------------------------------------------------------------------------ */

/* Edge e (weight w_e) is sampled once every w_max / w_e epochs: it is active
 * in epoch n when floor((n + 1) / eps_e) exceeds floor(n / eps_e), in fp32. */
int orc_active(float eps, int32_t epoch)
{
    float now = floorf((float)(epoch + 1) / eps);
    float before = floorf((float)epoch / eps);
    return now > before;
}

/* Ingest of the symmetric COO graph B (sparse-data handling section: a COO
 * sorted by row with a CSR index).  Drops entries with val <= 0 and self
 * loops; w_max is the largest remaining value; entries with
 * val < w_max / n_epochs are pruned (they would be sampled less than once).
 * The kept entries are sorted by (row, col); eps_e = w_max / val_e.
 * Status: 0 ok; -1 invalid (index out of range, non-finite value, a kept
 * (row, col) listed twice); -2 asymmetric (a kept (i, j, v) without a kept
 * (j, i) of bit-equal value).  Returns the kept count (or the status). */
int64_t orc_prep(int64_t n, const int32_t *rows, const int32_t *cols, const float *vals, int64_t nnz,
                 int32_t n_epochs, int64_t *row_ptr, int32_t *col, float *eps, float *w_max_out)
{
    for (int64_t t = 0; t < nnz; ++t) {
        if (rows[t] < 0 || rows[t] >= n || cols[t] < 0 || cols[t] >= n) return -1;
        if (!isfinite(vals[t])) return -1;
    }
    float w_max = 0.0f;
    for (int64_t t = 0; t < nnz; ++t)
        if (vals[t] > 0.0f && rows[t] != cols[t] && vals[t] > w_max) w_max = vals[t];
    float thresh = w_max / (float)n_epochs;
    float *val = malloc(sizeof(float) * (size_t)(nnz > 0 ? nnz : 1));
    if (!val) return -1;
    for (int64_t i = 0; i <= n; ++i) row_ptr[i] = 0;
    for (int64_t t = 0; t < nnz; ++t)
        if (vals[t] > 0.0f && rows[t] != cols[t] && vals[t] >= thresh) row_ptr[rows[t] + 1]++;
    for (int64_t i = 0; i < n; ++i) row_ptr[i + 1] += row_ptr[i];
    int64_t kept = row_ptr[n];
    int64_t *fill = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    for (int64_t i = 0; i < n; ++i) fill[i] = row_ptr[i];
    for (int64_t t = 0; t < nnz; ++t)
        if (vals[t] > 0.0f && rows[t] != cols[t] && vals[t] >= thresh) {
            int64_t p = fill[rows[t]]++;
            col[p] = cols[t];
            val[p] = vals[t];
        }
    free(fill);
    int64_t status = 0;
    for (int64_t i = 0; i < n && status == 0; ++i) {
        for (int64_t p = row_ptr[i] + 1; p < row_ptr[i + 1]; ++p) {
            int32_t c = col[p];
            float v = val[p];
            int64_t q = p - 1;
            while (q >= row_ptr[i] && col[q] > c) { col[q + 1] = col[q]; val[q + 1] = val[q]; --q; }
            col[q + 1] = c; val[q + 1] = v;
        }
        for (int64_t p = row_ptr[i] + 1; p < row_ptr[i + 1]; ++p)
            if (col[p] == col[p - 1]) status = -1;
    }
    for (int64_t i = 0; i < n && status == 0; ++i)
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            int32_t j = col[p];
            int64_t lo = row_ptr[j], hi = row_ptr[j + 1];
            while (lo < hi) { int64_t mid = (lo + hi) / 2; if (col[mid] < (int32_t)i) lo = mid + 1; else hi = mid; }
            uint32_t b1, b2;
            memcpy(&b1, &val[p], 4);
            if (lo < row_ptr[j + 1] && col[lo] == (int32_t)i) memcpy(&b2, &val[lo], 4);
            if (!(lo < row_ptr[j + 1] && col[lo] == (int32_t)i) || b1 != b2) { status = -2; break; }
        }
    if (status == 0)
        for (int64_t p = 0; p < kept; ++p) eps[p] = w_max / val[p];
    free(val);
    if (w_max_out) *w_max_out = w_max;
    return status != 0 ? status : kept;
}

/* ------------------------------------------------------------------------ */
/* Layout: epoch-synchronous (Jacobi) SGD over the edges of B, fp64.         */
/* ------------------------------------------------------------------------ */

typedef struct {
    double a, b;
    int32_t n_epochs;
    int32_t neg_rate;
} orc_params;

static const double ORC_CLIP = 4.0;      /* per-component gradient clip        */
static const double ORC_GAMMA = 1.0;     /* repulsion strength                 */
static const double ORC_REP_EPS = 1e-3;  /* regulariser added to d^2 in repulsion */

static double clip4(double g) { return g < -ORC_CLIP ? -ORC_CLIP : (g > ORC_CLIP ? ORC_CLIP : g); }

/* Attraction (gradient of log Phi, Phi = 1/(1 + a d^(2b))): coefficient on
 * (y_i - y_j); 0 when the points coincide. */
double orc_attr_coef(double d2, double a, double b)
{
    if (!(d2 > 0.0)) return 0.0;
    return -2.0 * a * b * pow(d2, b - 1.0) / (1.0 + a * pow(d2, b));
}

/* Repulsion (gradient of log(1 - Phi), with d^2 regularised by 1e-3):
 * coefficient on (y_i - y_k); 0 when the points coincide. */
double orc_rep_coef(double d2, double a, double b)
{
    if (!(d2 > 0.0)) return 0.0;
    return 2.0 * ORC_GAMMA * b / ((ORC_REP_EPS + d2) * (1.0 + a * pow(d2, b)));
}

/* Apply edge e = (i -> j) of epoch `epoch` to the accumulator D in push form:
 * y_i moves by +alpha g, y_j by -alpha g (both endpoints), then neg_rate
 * vertices k drawn uniformly move y_i alone (a draw equal to i is skipped). */
static void push_edge(const orc_params *P, int32_t dim, int64_t n, uint64_t seed, int32_t epoch,
                      double alpha, int64_t e, int64_t i, int64_t j, const double *E, double *D)
{
    double d2 = 0.0;
    for (int32_t d = 0; d < dim; ++d) {
        double df = E[i * dim + d] - E[j * dim + d];
        d2 += df * df;
    }
    double c = orc_attr_coef(d2, P->a, P->b);
    for (int32_t d = 0; d < dim; ++d) {
        double g = clip4(c * (E[i * dim + d] - E[j * dim + d]));
        D[i * dim + d] += alpha * g;
        D[j * dim + d] -= alpha * g;
    }
    for (int32_t r = 0; r < P->neg_rate; ++r) {
        int64_t kv = orc_negative_vertex(seed, e, epoch, r, n);
        if (kv == i) continue;
        double q2 = 0.0;
        for (int32_t d = 0; d < dim; ++d) {
            double df = E[i * dim + d] - E[kv * dim + d];
            q2 += df * df;
        }
        double cr = orc_rep_coef(q2, P->a, P->b);
        for (int32_t d = 0; d < dim; ++d) D[i * dim + d] += alpha * clip4(cr * (E[i * dim + d] - E[kv * dim + d]));
    }
}

#define ORC_CHUNKS 16

/* One epoch: every read uses the snapshot E; the summed updates are applied
 * at the end (the fp64 end-of-epoch mode of the reproducibility section).
 * alpha = 1 - epoch / n_epochs.  The edges are split into ORC_CHUNKS fixed
 * row ranges with private fp64 accumulators reduced in chunk order, so the
 * result does not depend on the thread count.  Returns the active count. */
int64_t orc_epoch(int64_t n, int32_t dim, const int64_t *row_ptr, const int32_t *col, const float *eps,
                  double a, double b, int32_t n_epochs, int32_t neg_rate, uint64_t seed, int32_t epoch,
                  const double *E, double *E_out)
{
    orc_params P = {a, b, n_epochs, neg_rate};
    const double alpha = 1.0 - (double)epoch / (double)n_epochs;
    const size_t sz = (size_t)n * (size_t)dim;
    double *D = calloc(sz * ORC_CHUNKS, sizeof(double));
    int64_t active[ORC_CHUNKS] = {0};
#pragma omp parallel for schedule(dynamic, 1)
    for (int ch = 0; ch < ORC_CHUNKS; ++ch) {
        int64_t r0 = n * ch / ORC_CHUNKS, r1 = n * (ch + 1) / ORC_CHUNKS;
        double *Dc = D + sz * (size_t)ch;
        for (int64_t i = r0; i < r1; ++i)
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
                if (orc_active(eps[e], epoch)) {
                    push_edge(&P, dim, n, seed, epoch, alpha, e, i, col[e], E, Dc);
                    active[ch]++;
                }
    }
    int64_t total = 0;
    for (int ch = 0; ch < ORC_CHUNKS; ++ch) total += active[ch];
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < (int64_t)sz; ++t) {
        double s = 0.0;
        for (int ch = 0; ch < ORC_CHUNKS; ++ch) s += D[sz * (size_t)ch + (size_t)t];
        E_out[t] = E[t] + s;
    }
    free(D);
    return total;
}

/* The update that lands on each vertex of `which` in one epoch, in push form
 * restricted to those targets: its own active out-edges (+alpha g and the
 * negatives) and the active edges (j -> i) that end on it (-alpha g).  The
 * in-edges are found through symmetry (the graph must be symmetric). */
void orc_epoch_rows(int64_t n, int32_t dim, const int64_t *row_ptr, const int32_t *col, const float *eps,
                    double a, double b, int32_t n_epochs, int32_t neg_rate, uint64_t seed, int32_t epoch,
                    const double *E, int64_t count, const int64_t *which, double *delta)
{
    orc_params P = {a, b, n_epochs, neg_rate};
    const double alpha = 1.0 - (double)epoch / (double)n_epochs;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < count; ++t) {
        int64_t i = which[t];
        double acc[64]; /* dim <= 64 */
        for (int32_t d = 0; d < dim; ++d) acc[d] = 0.0;
        /* own out-edges: the +alpha g share of the attraction and the negatives */
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            if (!orc_active(eps[e], epoch)) continue;
            int64_t j = col[e];
            double d2 = 0.0;
            for (int32_t d = 0; d < dim; ++d) { double df = E[i * dim + d] - E[j * dim + d]; d2 += df * df; }
            double c = orc_attr_coef(d2, P.a, P.b);
            for (int32_t d = 0; d < dim; ++d) acc[d] += alpha * clip4(c * (E[i * dim + d] - E[j * dim + d]));
            for (int32_t r = 0; r < P.neg_rate; ++r) {
                int64_t kv = orc_negative_vertex(seed, e, epoch, r, n);
                if (kv == i) continue;
                double q2 = 0.0;
                for (int32_t d = 0; d < dim; ++d) { double df = E[i * dim + d] - E[kv * dim + d]; q2 += df * df; }
                double cr = orc_rep_coef(q2, P.a, P.b);
                for (int32_t d = 0; d < dim; ++d) acc[d] += alpha * clip4(cr * (E[i * dim + d] - E[kv * dim + d]));
            }
        }
        /* in-edges (j -> i): edge id found in row j by binary search */
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            int64_t j = col[p];
            int64_t lo = row_ptr[j], hi = row_ptr[j + 1];
            while (lo < hi) { int64_t mid = (lo + hi) / 2; if (col[mid] < (int32_t)i) lo = mid + 1; else hi = mid; }
            if (lo >= row_ptr[j + 1] || col[lo] != (int32_t)i) continue;
            if (!orc_active(eps[lo], epoch)) continue;
            double d2 = 0.0;
            for (int32_t d = 0; d < dim; ++d) { double df = E[j * dim + d] - E[i * dim + d]; d2 += df * df; }
            double c = orc_attr_coef(d2, P.a, P.b);
            for (int32_t d = 0; d < dim; ++d) acc[d] -= alpha * clip4(c * (E[j * dim + d] - E[i * dim + d]));
        }
        for (int32_t d = 0; d < dim; ++d) delta[t * dim + d] = acc[d];
    }
}

/* Full layout: random init from `seed`, then epochs 0 .. n_epochs-1.
 * E_out (n x dim, fp64) receives the final layout; active_out (n_epochs) the
 * active edge count of each epoch (may be NULL). */
int orc_run(int64_t n, int32_t dim, const int64_t *row_ptr, const int32_t *col, const float *eps,
            double a, double b, int32_t n_epochs, int32_t neg_rate, uint64_t seed,
            double *E_out, int64_t *active_out)
{
    const size_t sz = (size_t)n * (size_t)dim;
    float *E0 = malloc(sizeof(float) * (sz ? sz : 1));
    double *tmp = malloc(sizeof(double) * (sz ? sz : 1));
    if (!E0 || !tmp) { free(E0); free(tmp); return -1; }
    orc_init(n, dim, seed, E0);
    for (size_t t = 0; t < sz; ++t) E_out[t] = (double)E0[t];
    for (int32_t ep = 0; ep < n_epochs; ++ep) {
        int64_t act = orc_epoch(n, dim, row_ptr, col, eps, a, b, n_epochs, neg_rate, seed, ep, E_out, tmp);
        memcpy(E_out, tmp, sizeof(double) * sz);
        if (active_out) active_out[ep] = act;
    }
    free(E0);
    free(tmp);
    return 0;
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of later parallel regions (the sums are reduced in a fixed chunk
 * order, so the results do not depend on it). */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
