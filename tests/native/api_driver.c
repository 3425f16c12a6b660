/*
 * api_driver.c -- test driver for the host side of the C-ABI library, for
 * builds whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer.
 * It needs no GPU: every call below fails in argument checking or at device
 * discovery, before any kernel launch.  Exit status 0 when each call returns
 * the documented error code and message.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "umap_layout.h"

static int failures = 0;

static void expect(int got, int want, const char *needle, const char *what)
{
    const char *msg = umap_layout_last_error();
    if (got != want || (needle && !strstr(msg, needle))) {
        fprintf(stderr, "%s: got %d (%s), want %d (%s)\n", what, got, msg, want, needle ? needle : "-");
        ++failures;
    }
}

int main(void)
{
    enum { N = 64, NNZ = 128 };
    /* exact-size heap buffers: a read past their end is reported */
    int32_t *rows = malloc(sizeof(int32_t) * NNZ);
    int32_t *cols = malloc(sizeof(int32_t) * NNZ);
    float *vals = malloc(sizeof(float) * NNZ);
    float *table = malloc(sizeof(float) * N * 2);
    for (int t = 0; t < NNZ; ++t) {
        rows[t] = t % N;
        cols[t] = (t + 1 + t / N) % N;
        vals[t] = 0.5f;
    }
    for (int t = 0; t < 2 * N; ++t) table[t] = (float)t;
    umap_layout *h = (umap_layout *)0x1;

    expect(umap_layout_create(NULL, N, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL, "NULL", "out");
    expect(umap_layout_create(&h, 0, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL, "n must", "n");
    if (h != NULL) {
        fprintf(stderr, "out not cleared on failure\n");
        ++failures;
    }
    expect(umap_layout_create(&h, N, 17, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL, "n_components",
           "dim");
    expect(umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, NAN, 0.9f, 10, 5), UMAP_E_INVAL, "a must", "a");
    expect(umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, 1.5f, -1.0f, 10, 5), UMAP_E_INVAL, "b must", "b");
    expect(umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 0, 5), UMAP_E_INVAL, "n_epochs", "epochs");
    expect(umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, -1), UMAP_E_INVAL, "neg_rate", "rate");
    expect(umap_layout_create(&h, N, 2, NULL, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL, "NULL", "rows");
    cols[NNZ - 1] = N;   /* the last entry is the one out of range: the whole input is scanned */
    expect(umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL, "outside", "index");
    cols[NNZ - 1] = 0;
    vals[NNZ - 1] = INFINITY;
    expect(umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL, "finite", "value");
    vals[NNZ - 1] = 0.5f;

    expect(umap_transform_create(&h, N, 2, table, 0, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL,
           "n_table", "n_table");
    expect(umap_transform_create(&h, N, 2, NULL, N, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL,
           "table is NULL", "table");
    table[2 * N - 1] = NAN;   /* last table entry */
    expect(umap_transform_create(&h, N, 2, table, N, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL,
           "table entry", "table value");
    table[2 * N - 1] = 0.0f;
    cols[NNZ - 1] = N;
    expect(umap_transform_create(&h, N, 2, table, N, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5), UMAP_E_INVAL,
           "outside", "transform index");
    cols[NNZ - 1] = 0;
    expect(umap_layout_create_device(&h, N, 2, NULL, NULL, NULL, NNZ, 1.5f, 0.9f, 10, 5, NULL), UMAP_E_INVAL, "NULL",
           "device inputs");

    /* valid arguments on a host without a GPU: device discovery fails cleanly */
    int rc = umap_layout_create(&h, N, 2, rows, cols, vals, NNZ, 1.5f, 0.9f, 10, 5);
    if (rc == UMAP_OK) {
        umap_layout_destroy(h);   /* a GPU is present: nothing more to check here */
    } else {
        expect(rc, UMAP_E_DEVICE, "device", "no device");
        if (h != NULL) {
            fprintf(stderr, "out not cleared after a device failure\n");
            ++failures;
        }
    }

    /* handle-free checks */
    expect(umap_layout_init(NULL, 1), UMAP_E_INVAL, "NULL", "init");
    expect(umap_layout_run(NULL, 1), UMAP_E_INVAL, "NULL", "run");
    expect(umap_layout_run_epochs(NULL, 1, 0, 1), UMAP_E_INVAL, "NULL", "run_epochs");
    expect(umap_layout_get(NULL, table), UMAP_E_INVAL, "NULL", "get");
    expect(umap_layout_get_device(NULL, table), UMAP_E_INVAL, "NULL", "get_device");
    expect(umap_layout_set_embedding(NULL, table), UMAP_E_INVAL, "NULL", "set_embedding");
    expect(umap_layout_get_graph(NULL, NULL, NULL, NULL, NULL), UMAP_E_INVAL, "NULL", "get_graph");
    expect(umap_layout_stats(NULL, NULL), UMAP_E_INVAL, "NULL", "stats");
    expect(umap_layout_set_stream(NULL, NULL), UMAP_E_INVAL, "NULL", "set_stream");
    expect(umap_layout_set_kernel(NULL, 0), UMAP_E_INVAL, "NULL", "set_kernel");
    expect(umap_layout_set_mode(NULL, 0), UMAP_E_INVAL, "NULL", "set_mode");
    expect(umap_layout_set_rows(NULL, 0, 1), UMAP_E_INVAL, "NULL", "set_rows");
    expect(umap_layout_debug_active(NULL, 0, NULL), UMAP_E_INVAL, "NULL", "debug_active");
    expect(umap_layout_debug_negatives(NULL, 1, 0, 0, 1, NULL), UMAP_E_INVAL, "NULL", "debug_negatives");
    umap_layout_destroy(NULL);

    expect(umap_fuzzy_graph_device(N, 0, rows, vals, rows, cols, vals, NULL), UMAP_E_INVAL, "k must", "graph k");
    expect(umap_fuzzy_graph_device(N, 4, NULL, vals, rows, cols, vals, NULL), UMAP_E_INVAL, "NULL", "graph ptr");
    expect(umap_trustworthiness(table, N, 2, table, 2, 0, NULL, NULL), UMAP_E_INVAL, "NULL", "trust out");
    double tw = 0.0;
    expect(umap_trustworthiness(table, N, 2, table, 2, 65, &tw, NULL), UMAP_E_INVAL, "k must", "trust k");
    expect(umap_trustworthiness(table, 4, 2, table, 2, 3, &tw, NULL), UMAP_E_INVAL, "2n - 3k - 1", "trust n");
    expect(umap_probe_copy(table, table, 15, NULL), UMAP_E_INVAL, "16", "probe copy");
    expect(umap_probe_gather(table, 3, 256, 1, table, NULL), UMAP_E_INVAL, "power of two", "probe gather");

    /* the curve fit is host code end to end */
    float a = 0.0f, b = 0.0f;
    expect(umap_fit_ab(1.0f, 0.1f, &a, &b), UMAP_OK, NULL, "fit_ab");
    if (!(fabsf(a - 1.577f) < 0.01f && fabsf(b - 0.895f) < 0.01f)) {
        fprintf(stderr, "fit_ab(1, 0.1) = (%g, %g)\n", a, b);
        ++failures;
    }
    expect(umap_fit_ab(1.0f, -0.5f, &a, &b), UMAP_E_INVAL, NULL, "fit_ab min_dist");

    free(rows);
    free(cols);
    free(vals);
    free(table);
    if (failures) return 1;
    printf("api driver ok\n");
    return 0;
}
