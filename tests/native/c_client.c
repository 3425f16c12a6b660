/*
 * c_client.c -- a plain C program using the layout library through its C ABI
 * (no Python): builds a symmetric ring graph, lays it out twice with one seed
 * and once with the other kernel, and checks that the three layouts agree bit
 * for bit, that the sampled-edge count matches the schedule, and that a bad
 * call reports UMAP_E_INVAL with a message.  Exit status 0 on success; 77 when
 * no GPU is present.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "umap_layout.h"

#define CHECK(c)                                                                        \
    do {                                                                                \
        if (!(c)) {                                                                     \
            fprintf(stderr, "check failed: %s (line %d): %s\n", #c, __LINE__,           \
                    umap_layout_last_error());                                          \
            return 1;                                                                   \
        }                                                                               \
    } while (0)

int main(void)
{
    enum { N = 20000, HALF = 7, EPOCHS = 60, R = 5 };
    const int64_t nnz = (int64_t)N * 2 * HALF;
    int32_t *rows = malloc(sizeof(int32_t) * nnz), *cols = malloc(sizeof(int32_t) * nnz);
    float *vals = malloc(sizeof(float) * nnz);
    int64_t t = 0;
    for (int32_t i = 0; i < N; ++i)
        for (int32_t s = 1; s <= HALF; ++s) {
            /* (i, i + s) and (i + s, i) with the same weight, ring-wise */
            const int32_t j = (i + s) % N;
            const float w = 1.0f / (float)s;
            rows[t] = i, cols[t] = j, vals[t] = w, ++t;
            rows[t] = j, cols[t] = i, vals[t] = w, ++t;
        }
    float a = 0.0f, b = 0.0f;
    CHECK(umap_fit_ab(1.0f, 0.1f, &a, &b) == UMAP_OK);

    umap_layout *h = NULL;
    int rc = umap_layout_create(&h, N, 2, rows, cols, vals, nnz, a, b, EPOCHS, R);
    if (rc == UMAP_E_DEVICE) {
        printf("no GPU: %s\n", umap_layout_last_error());
        return 77;
    }
    CHECK(rc == UMAP_OK && h != NULL);
    float *y0 = malloc(sizeof(float) * N * 2), *y1 = malloc(sizeof(float) * N * 2);
    CHECK(umap_layout_run(h, 42) == UMAP_OK);
    CHECK(umap_layout_get(h, y0) == UMAP_OK);
    umap_layout_stats_t st;
    CHECK(umap_layout_stats(h, &st) == UMAP_OK);
    CHECK(st.nnz_kept > 0 && st.nnz_kept <= nnz && st.epochs_done == EPOCHS);
    CHECK(st.edge_updates == st.active_edges * (1 + R));

    /* the schedule, counted on the host from the kept graph, gives the same count */
    int64_t *row_ptr = malloc(sizeof(int64_t) * (N + 1));
    int32_t *col = malloc(sizeof(int32_t) * st.nnz_kept);
    float *eps = malloc(sizeof(float) * st.nnz_kept);
    int64_t kept = 0;
    CHECK(umap_layout_get_graph(h, row_ptr, col, eps, &kept) == UMAP_OK && kept == st.nnz_kept);
    int64_t sampled = 0;
    for (int64_t e = 0; e < kept; ++e)
        for (int32_t ep = 0; ep < EPOCHS; ++ep)
            sampled += floorf((float)(ep + 1) / eps[e]) > floorf((float)ep / eps[e]);
    CHECK(sampled == st.active_edges);

    CHECK(umap_layout_run(h, 42) == UMAP_OK);
    CHECK(umap_layout_get(h, y1) == UMAP_OK);
    CHECK(memcmp(y0, y1, sizeof(float) * N * 2) == 0);
    CHECK(umap_layout_set_kernel(h, 1) == UMAP_OK);
    CHECK(umap_layout_run(h, 42) == UMAP_OK);
    CHECK(umap_layout_get(h, y1) == UMAP_OK);
    CHECK(memcmp(y0, y1, sizeof(float) * N * 2) == 0);
    for (int64_t k = 0; k < (int64_t)N * 2; ++k) CHECK(isfinite(y0[k]));

    CHECK(umap_layout_run_epochs(h, 42, 5, 4) == UMAP_E_INVAL);
    CHECK(strstr(umap_layout_last_error(), "first") != NULL);
    umap_layout_destroy(h);
    printf("c client ok: %lld kept edges, %lld sampled, %.2f ms of epochs\n", (long long)kept,
           (long long)sampled, st.epochs_ms);
    free(rows), free(cols), free(vals), free(y0), free(y1), free(row_ptr), free(col), free(eps);
    return 0;
}
