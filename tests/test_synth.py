"""The seeded input generators (shared by the oracle and the GPU path) do what
their recipes state: same seed, same arrays; window kNN lists hold k distinct
neighbours from the +-64 window inside the vertex's cluster, never the vertex,
with increasing distances; cluster bounds cover 0..n with the stated sizes."""

import numpy as np

from paper_2008_00325_amd import synth


def test_window_knn_recipe():
    n, k = 20_000, 15
    bounds = synth.cluster_bounds(n, 7)
    ids, dist = synth.window_knn(n, k, bounds, seed=3)
    ids2, dist2 = synth.window_knn(n, k, bounds, seed=3)
    assert np.array_equal(ids, ids2) and np.array_equal(dist, dist2)
    assert not np.array_equal(ids, synth.window_knn(n, k, bounds, seed=4)[0])
    rows = np.arange(n)[:, None]
    cl = np.searchsorted(bounds, np.arange(n), side="right") - 1
    lo, hi = bounds[cl][:, None], bounds[cl + 1][:, None]
    assert np.all(np.abs(ids - rows) <= synth.WINDOW) and np.all(ids != rows)
    assert np.all((ids >= lo) & (ids < hi))
    srt = np.sort(ids, axis=1)
    assert np.all(np.diff(srt, axis=1) > 0)                  # distinct
    assert np.all(np.diff(dist, axis=1) > 0) and np.all(dist > 0)
    # progress reports do not change the draws
    seen = []
    ids3, _ = synth.window_knn(n, k, bounds, seed=3, progress=seen.append)
    assert np.array_equal(ids, ids3) and seen[-1] == n


def test_cluster_bounds():
    b = synth.cluster_bounds(1000, 7)
    assert b[0] == 0 and b[-1] == 1000 and np.all(np.diff(b) >= 142)
    b = synth.cluster_bounds(100_000, 30, lognormal_sigma=1.0, seed=5)
    sizes = np.diff(b)
    assert b[0] == 0 and b[-1] == 100_000 and sizes.min() >= 2 * synth.WINDOW + 1
    assert sizes.max() > 3 * sizes.min()                       # log-normal spread


def test_points_and_states():
    X, lab = synth.blobs(1000, 16, 5, seed=1)
    assert X.shape == (1000, 16) and X.dtype == np.float32 and np.bincount(lab).tolist() == [200] * 5
    assert np.array_equal(X, synth.blobs(1000, 16, 5, seed=1)[0])
    Xi, _ = synth.image_like(500, 784, 10, seed=2)
    assert Xi.min() >= 0.0 and Xi.max() <= 1.0
    E = synth.embedding_state(100, 3, 9, 5.0)
    assert E.dtype == np.float32 and np.all(np.abs(E) <= 5.0)


def test_transform_graph_recipe():
    rows, cols, vals = synth.transform_graph(3000, 10_000, k=15, seed=6)
    assert rows.size == cols.size == vals.size == 3000 * 15
    assert np.all(np.diff(rows) >= 0) and np.all((cols >= 0) & (cols < 10_000))
    c = cols.reshape(3000, 15)
    assert np.all(np.diff(np.sort(c, axis=1), axis=1) > 0)     # distinct per point
    assert np.all(c.max(axis=1) - c.min(axis=1) <= 2 * synth.WINDOW)
    assert np.all((vals >= 0.05) & (vals < 1.0))


def test_random_symmetric_coo():
    r, c, v = synth.random_symmetric_coo(500, 8, seed=3)
    pairs = dict(zip(zip(r.tolist(), c.tolist()), v.tolist()))
    assert len(pairs) == r.size and np.all(r != c)
    for (i, j), w in pairs.items():
        assert pairs[(j, i)] == w
