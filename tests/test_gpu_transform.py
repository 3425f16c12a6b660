"""GPU parity of the transform (new points laid out against a frozen trained
layout; only the new points move -- embedding-updates section) against the
oracle, through the C ABI:
  * the bipartite graph (row_ptr, col, eps): bit-exact;
  * the initial layout (weighted mean of the kept neighbours): <= 1e-5;
  * one epoch fed the same fp32 state: max |GPU - oracle| <= 1e-4, both epoch
    kernels, tables of one and of four ranges;
  * a full transform against the oracle's own trained layout: kNN-label
    accuracy and trustworthiness of the new points within 0.01 of the
    oracle's transform.
"""

import sys

import numpy as np
import pytest

import oracle as O
from paper_2008_00325_amd import synth
from paper_2008_00325_amd import umap_layout as U

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def torch_device_first():
    """Initialise torch's HIP runtime before the library's."""
    import torch

    torch.cuda.init()
    torch.cuda.set_device(0)


def case(msg):
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def _membership_graph(Q, X, k):
    """Weights of the new points' kNN among the training points (Eq. 1), no union."""
    ids, dist = O.exact_knn_cross(Q, X, k)
    rho, sigma = O.smooth_knn(dist)
    A = O.membership(dist, rho, sigma)
    rows = np.repeat(np.arange(Q.shape[0], dtype=np.int32), k)
    return rows, ids.ravel().astype(np.int32), A.ravel().astype(np.float32)


def _split_blobs(n_all=2600, n_new=600, seed=11):
    X_all, lab = synth.blobs(n_all, 16, 5, seed=seed)
    perm = np.random.default_rng(seed + 1).permutation(n_all)
    tr, nw = perm[: n_all - n_new], perm[n_all - n_new:]
    return X_all[tr], lab[tr], X_all[nw], lab[nw]


def _check_graph(h, g):
    row_ptr, col, eps = U.umap_layout_get_graph(h)
    assert np.array_equal(row_ptr, g.row_ptr)
    assert np.array_equal(col, g.col)
    assert np.array_equal(eps.view(np.uint32), g.eps.view(np.uint32))


def _epoch_parity(h, g, T, states, epochs, a, b, N, R, seed, what):
    for kernel in (0, 1):
        U.umap_layout_set_kernel(h, kernel)
        for s, E in enumerate(states):
            for ep in epochs:
                case(f"{what}: kernel {kernel} state {s} epoch {ep}")
                U.umap_layout_set_embedding(h, E)
                U.umap_layout_run_epochs(h, seed, ep, ep + 1)
                got = U.umap_layout_get(h)
                ref, act = O.frozen_epoch(g, E, T, ep, a, b, N, R, seed)
                err = float(np.abs(got.astype(np.float64) - ref).max())
                print(f"  max|diff| = {err:.3e}  active = {act}", flush=True)
                assert err <= TOL
                assert U.umap_layout_stats(h)["active_edges"] == act


def test_transform_graph_init_and_epoch_parity():
    X, _, Q, _ = _split_blobs()
    T = synth.embedding_state(X.shape[0], 2, 8, 10.0)
    r, c, v = _membership_graph(Q, X, 15)
    N, R = 100, 5
    a, b = O.fit_ab(1.0, 0.1)
    g = O.prep_bipartite(Q.shape[0], X.shape[0], r, c, v, N)
    with U.umap_transform_create(Q.shape[0], T, r, c, v, a, b, N, R) as h:
        _check_graph(h, g)
        U.umap_layout_init(h, 7)
        Y0 = U.umap_layout_get(h)
        ref0 = O.transform_init(g, T)
        assert float(np.abs(Y0 - ref0).max()) <= 1e-5
        states = [Y0, synth.embedding_state(Q.shape[0], 2, 9, 10.0)]
        _epoch_parity(h, g, T, states, (0, 1, N // 2, N - 1), a, b, N, R, 5, "blobs transform")
        with pytest.raises(U.UmapLayoutError) as ei:
            U.umap_layout_set_mode(h, U.UMAP_MODE_ASYNC)
            U.umap_layout_run(h, 1)
        assert ei.value.code == U.UMAP_E_INVAL


@pytest.mark.parametrize("n_table,dim,ranges", [(1_000_000, 2, 4), (700_000, 3, 4), (120_000, 16, 4),
                                                (400_000, 3, 1), (50_000, 16, 2)])
def test_transform_epoch_parity_large_table(n_table, dim, ranges):
    """Large tables: several ranges (the negative samples are filed by range),
    one range of 4.8 MB (each repulsion applied by the draw kernel), or two
    ranges of a 3.2 MB table at 16 components (one range only up to 2 MB at
    that width): 50,003 new points with 15 edges each to scattered table rows."""
    n_new, k = 50_003, 15
    rng = np.random.default_rng(n_table + dim)
    start = rng.integers(0, n_table, size=(n_new, 1))
    stride = rng.integers(1, n_table // k, size=(n_new, 1))
    cols = ((start + stride * np.arange(k)) % n_table).astype(np.int32).ravel()
    rows = np.repeat(np.arange(n_new, dtype=np.int32), k)
    vals = rng.uniform(0.05, 1.0, size=rows.size).astype(np.float32)
    T = synth.embedding_state(n_table, dim, 12, 10.0)
    N, R = 60, 5
    a, b = O.fit_ab(1.0, 0.1)
    g = O.prep_bipartite(n_new, n_table, rows, cols, vals, N)
    with U.umap_transform_create(n_new, T, rows, cols, vals, a, b, N, R) as h:
        _check_graph(h, g)
        assert U.umap_layout_stats(h)["table_ranges"] == ranges
        # negatives are drawn from the table's rows
        got = U.umap_layout_debug_negatives(h, 9, 7, 1000, 5000)
        assert np.array_equal(got, O.negative_vertices(9, 7, 1000, 5000, R, n_table))
        states = [synth.embedding_state(n_new, dim, 13, 10.0)]
        _epoch_parity(h, g, T, states, (0, N // 2, N - 1), a, b, N, R, 9, f"table {n_table} x {dim}")


def _label_accuracy(Y, T, lab_train, lab_new, k=15):
    from scipy.spatial import cKDTree

    _, nb = cKDTree(np.asarray(T, np.float64)).query(np.asarray(Y, np.float64), k=k)
    votes = lab_train[nb]
    pred = np.array([np.bincount(row, minlength=lab_train.max() + 1).argmax() for row in votes])
    return float((pred == lab_new).mean())


def test_transform_quality_blobs():
    """Fit the training points with the oracle, then lay out the new points
    against that frozen layout on the GPU and with the oracle."""
    X, lab_x, Q, lab_q = _split_blobs()
    a, b = O.fit_ab(1.0, 0.1)
    ids, dist = O.exact_knn(X, 15)
    rf, cf, vf = O.fuzzy_graph(ids, dist)
    gf = O.prep(X.shape[0], rf, cf, vf, 200)
    case("oracle fit of the training points")
    T = O.run(gf, 2, a, b, 200, 5, 3)[0].astype(np.float32)
    r, c, v = _membership_graph(Q, X, 15)
    N, R, seed = 100, 5, 4
    g = O.prep_bipartite(Q.shape[0], X.shape[0], r, c, v, N)
    case("GPU transform")
    with U.umap_transform_create(Q.shape[0], T, r, c, v, a, b, N, R) as h:
        U.umap_layout_run(h, seed)
        Yg = U.umap_layout_get(h)
        st = U.umap_layout_stats(h)
    case("oracle transform")
    Yo, act = O.transform_run(g, T, a, b, N, R, seed)
    assert st["active_edges"] == int(act.sum())
    assert np.all(np.isfinite(Yg))
    acc_g = _label_accuracy(Yg, T, lab_x, lab_q)
    acc_o = _label_accuracy(Yo, T, lab_x, lab_q)
    tg = O.trustworthiness(Q, Yg, 15)
    to = O.trustworthiness(Q, Yo, 15)
    print(f"  accuracy {acc_g:.4f} (oracle {acc_o:.4f}); T@15 {tg:.5f} (oracle {to:.5f})", flush=True)
    assert acc_g >= 0.95
    assert abs(acc_g - acc_o) <= 0.01
    assert abs(tg - to) <= 0.01


def test_transform_edge_cases():
    """New points without kept edges start at the origin and never move; an
    empty graph leaves every new point at the origin; weights of zero are
    dropped."""
    T = synth.embedding_state(100, 2, 21, 10.0)
    a, b = O.fit_ab(1.0, 0.1)
    rows = np.array([0, 0, 3, 3, 3, 4], np.int32)
    cols = np.array([5, 7, 10, 11, 99, 50], np.int32)
    vals = np.array([1.0, 0.5, 0.25, 1.0, 0.75, 0.0], np.float32)   # row 4's only entry has weight 0
    g = O.prep_bipartite(5, 100, rows, cols, vals, 20)
    case("transform edge cases")
    with U.umap_transform_create(5, T, rows, cols, vals, a, b, 20, 5) as h:
        _check_graph(h, g)
        U.umap_layout_init(h, 3)
        assert float(np.abs(U.umap_layout_get(h) - O.transform_init(g, T)).max()) <= 1e-5
        U.umap_layout_run(h, 3)
        Y = U.umap_layout_get(h)
        assert np.all(np.isfinite(Y))
        assert np.array_equal(Y[[1, 2, 4]], np.zeros((3, 2), np.float32))
        assert U.umap_layout_stats(h)["nnz_kept"] == 5
    empty = np.zeros(0, np.int32)
    with U.umap_transform_create(3, T, empty, empty, np.zeros(0, np.float32), a, b, 10, 5) as h:
        U.umap_layout_run(h, 1)
        assert np.array_equal(U.umap_layout_get(h), np.zeros((3, 2), np.float32))
        assert U.umap_layout_stats(h)["active_edges"] == 0
