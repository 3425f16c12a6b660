/*
 * oracle_driver.c -- test driver that runs every routine of the CPU oracle on a
 * small synthetic graph, for builds with AddressSanitizer and
 * UndefinedBehaviorSanitizer.  Exit status 0 when the invariants hold.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
void orc_negative_batch(uint64_t seed, int32_t epoch, int64_t e_first, int64_t count, int32_t neg_rate, int64_t n,
                        uint32_t *out);
void orc_init(int64_t n, int32_t dim, uint64_t seed, float *out);
void orc_smooth_knn(int64_t n, int32_t k, const float *dists, double *rho, double *sigma);
void orc_membership(int64_t n, int32_t k, const float *dists, const double *rho, const double *sigma, double *A);
int64_t orc_fuzzy_union(int64_t n, int32_t k, const int32_t *ids, const double *A, int32_t *rows, int32_t *cols,
                        double *vals);
int orc_fit_ab(double spread, double min_dist, double *a_out, double *b_out);
int64_t orc_prep(int64_t n, const int32_t *rows, const int32_t *cols, const float *vals, int64_t nnz,
                 int32_t n_epochs, int64_t *row_ptr, int32_t *col, float *eps, float *w_max_out);
int64_t orc_epoch(int64_t n, int32_t dim, const int64_t *row_ptr, const int32_t *col, const float *eps, double a,
                  double b, int32_t n_epochs, int32_t neg_rate, uint64_t seed, int32_t epoch, const double *E,
                  double *E_out);
int orc_run(int64_t n, int32_t dim, const int64_t *row_ptr, const int32_t *col, const float *eps, double a, double b,
            int32_t n_epochs, int32_t neg_rate, uint64_t seed, double *E_out, int64_t *active_out);

#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                              \
        }                                                          \
    } while (0)

int main(void)
{
    enum { N = 300, K = 10, DIM = 3, EPOCHS = 30, R = 5 };
    /* kNN lists: neighbours at offsets 1..K to the right (cyclic), distances
     * growing with the offset; seeded by a small linear congruential generator */
    static int32_t ids[N * K];
    static float dist[N * K];
    uint32_t lcg = 12345u;
    for (int i = 0; i < N; ++i) {
        float d = 0.0f;
        for (int s = 0; s < K; ++s) {
            lcg = lcg * 1664525u + 1013904223u;
            d += 0.05f + (float)(lcg >> 8) / 16777216.0f;
            ids[i * K + s] = (i + 1 + s) % N;
            dist[i * K + s] = d;
        }
    }
    static double rho[N], sigma[N], A[N * K];
    orc_smooth_knn(N, K, dist, rho, sigma);
    orc_membership(N, K, dist, rho, sigma, A);
    for (int i = 0; i < N; ++i) {
        double s = 0.0;
        for (int t = 0; t < K; ++t) s += A[i * K + t];
        CHECK(fabs(s - log2((double)K)) < 1e-5 || sigma[i] > 0.0);
    }
    static int32_t rows[2 * N * K], cols[2 * N * K];
    static double vals[2 * N * K];
    int64_t m = orc_fuzzy_union(N, K, ids, A, rows, cols, vals);
    CHECK(m > 0 && m <= 2 * N * K);
    static float fv[2 * N * K];
    for (int64_t t = 0; t < m; ++t) fv[t] = (float)vals[t];
    static int64_t row_ptr[N + 1];
    static int32_t col[2 * N * K];
    static float eps[2 * N * K];
    float w_max = 0.0f;
    int64_t kept = orc_prep(N, rows, cols, fv, m, EPOCHS, row_ptr, col, eps, &w_max);
    CHECK(kept > 0 && kept <= m && row_ptr[N] == kept && w_max > 0.0f);
    double a = 0.0, b = 0.0;
    CHECK(orc_fit_ab(1.0, 0.1, &a, &b) == 0 && a > 1.5 && b > 0.85);
    static float E0[N * DIM];
    static double E[N * DIM], E1[N * DIM];
    orc_init(N, DIM, 7u, E0);
    for (int t = 0; t < N * DIM; ++t) E[t] = E0[t];
    int64_t act = orc_epoch(N, DIM, row_ptr, col, eps, a, b, EPOCHS, R, 7u, EPOCHS / 2, E, E1);
    CHECK(act >= 0 && act <= kept);
    for (int t = 0; t < N * DIM; ++t) CHECK(isfinite(E1[t]));
    static int64_t active[EPOCHS];
    CHECK(orc_run(N, DIM, row_ptr, col, eps, a, b, EPOCHS, R, 9u, E, active) == 0);
    for (int t = 0; t < N * DIM; ++t) CHECK(isfinite(E[t]));
    uint32_t neg[20 * R];
    orc_negative_batch(3u, 4, 0, 20, R, N, neg);
    for (int t = 0; t < 20 * R; ++t) CHECK(neg[t] < N);
    uint32_t ctr[4] = {1u, 2u, 3u, 4u}, key[2] = {5u, 6u}, o1[4], o2[4];
    orc_philox4x32_10(ctr, key, o1);
    orc_philox4x32_10(ctr, key, o2);
    for (int t = 0; t < 4; ++t) CHECK(o1[t] == o2[t]);
    /* an asymmetric graph is rejected without touching memory beyond its inputs */
    int32_t r2[1] = {0}, c2[1] = {1};
    float v2[1] = {1.0f};
    CHECK(orc_prep(N, r2, c2, v2, 1, EPOCHS, row_ptr, col, eps, &w_max) < 0);
    printf("oracle driver ok: %lld union entries, %lld kept\n", (long long)m, (long long)kept);
    return 0;
}
