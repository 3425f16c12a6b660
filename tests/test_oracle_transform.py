"""Pins of the oracle's transform (new points laid out against a frozen
trained layout; only the new points move -- embedding-updates section).

The transform epoch is written once, in numpy, with the attraction factor and
the table as parameters; with the table equal to the moving layout, factor 2
and self draws skipped it is the fit's epoch, which the C oracle computes by
an independent route (push form, both endpoints).  That reduction pins the
terms, signs and indices; the remaining pins cover what differs."""

import numpy as np
import pytest
from sklearn.neighbors import NearestNeighbors

from paper_2008_00325_amd import synth


def _sym_graph(orc, n=400, deg=8, seed=5, n_epochs=40):
    r, c, v = synth.random_symmetric_coo(n, deg, seed)
    return (r, c, v), orc.prep(n, r, c, v, n_epochs)


def test_prep_bipartite_equals_prep_on_a_symmetric_graph(orc):
    (r, c, v), g = _sym_graph(orc)
    gb = orc.prep_bipartite(g.n, g.n, r, c, v, 40)
    assert np.array_equal(gb.row_ptr, g.row_ptr)
    assert np.array_equal(gb.col, g.col)
    assert np.array_equal(gb.eps.view(np.uint32), g.eps.view(np.uint32))
    assert np.float32(gb.w_max) == np.float32(g.w_max)


def test_prep_bipartite_keeps_equal_indices_and_checks_inputs(orc):
    rows = np.array([0, 0, 1, 2], np.int32)
    cols = np.array([0, 3, 1, 4], np.int32)
    vals = np.array([1.0, 0.5, 0.25, 0.0], np.float32)
    g = orc.prep_bipartite(3, 5, rows, cols, vals, 4)
    # (0, 0) and (1, 1) are edges to table vertices 0 and 1; the zero weight goes
    assert list(g.row_ptr) == [0, 2, 3, 3]
    assert list(g.col) == [0, 3, 1]
    assert list(g.eps) == [1.0, 2.0, 4.0]
    with pytest.raises(orc.PrepError):
        orc.prep_bipartite(3, 4, rows, cols, vals, 4)        # column 4 outside the table
    with pytest.raises(orc.PrepError):
        orc.prep_bipartite(3, 5, rows, cols, np.array([1, np.nan, 1, 1], np.float32), 4)
    with pytest.raises(orc.PrepError):
        orc.prep_bipartite(3, 5, np.array([0, 0], np.int32), np.array([2, 2], np.int32),
                           np.array([1, 1], np.float32), 4)  # listed twice


@pytest.mark.parametrize("R", [0, 5])
def test_frozen_epoch_reduces_to_the_fit_epoch(orc, R):
    (r, c, v), g = _sym_graph(orc, n_epochs=40)
    a, b = orc.fit_ab(1.0, 0.1)
    E = synth.embedding_state(g.n, 3, 9, 5.0).astype(np.float64)
    for ep in (0, 1, 17, 39):
        ref, act_ref = orc.epoch(g, E, ep, a, b, 40, R, 21)
        got, act = orc.frozen_epoch(g, E, E, ep, a, b, 40, R, 21, attr_mult=2.0, self_skip=True)
        assert act == act_ref
        assert np.abs(got - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())


def test_frozen_epoch_moves_only_toward_the_table(orc):
    """One new point, one edge to a frozen vertex, no negatives: late in the run
    (small step) the point moves straight toward its neighbour; a point sitting
    on its only neighbour does not move."""
    T = np.array([[0.0, 0.0], [3.0, 4.0]])
    g = orc.prep_bipartite(2, 2, np.array([0, 1], np.int32), np.array([1, 1], np.int32),
                           np.array([1.0, 1.0], np.float32), 100)
    a, b = orc.fit_ab(1.0, 0.1)
    Y = np.array([[0.0, 0.0], [3.0, 4.0]])
    out, act = orc.frozen_epoch(g, Y, T, 99, a, b, 100, 0, 1)
    assert act == 2
    step = out[0] - Y[0]
    assert np.linalg.norm(out[0] - T[1]) < np.linalg.norm(Y[0] - T[1])
    assert abs(step[0] * 4.0 - step[1] * 3.0) < 1e-15      # along the line to (3, 4)
    assert np.array_equal(out[1], Y[1])


def test_transform_init_weighted_mean(orc):
    T = np.array([[1.0, 2.0], [5.0, -2.0], [9.0, 9.0]])
    rows = np.array([0, 1, 1], np.int32)
    cols = np.array([2, 0, 1], np.int32)
    vals = np.array([0.5, 1.0, 0.5], np.float32)
    g = orc.prep_bipartite(3, 3, rows, cols, vals, 2)
    Y = orc.transform_init(g, T)
    assert np.array_equal(Y[0], T[2])                        # one neighbour: its position
    assert np.allclose(Y[1], (T[0] * 1.0 + T[1] * 0.5) / 1.5, rtol=0, atol=1e-15)
    assert np.array_equal(Y[2], [0.0, 0.0])                  # no kept edge: the origin


def test_exact_knn_cross_matches_library(orc):
    X, _ = synth.blobs(800, 8, 4, seed=6)
    Q, _ = synth.blobs(150, 8, 4, seed=7)
    ids, dist = orc.exact_knn_cross(Q, X, 10, batch=64)
    nn = NearestNeighbors(n_neighbors=10, algorithm="brute").fit(X.astype(np.float64))
    d_ref, i_ref = nn.kneighbors(Q.astype(np.float64))
    assert np.array_equal(np.sort(ids, axis=1), np.sort(i_ref, axis=1))
    assert np.allclose(dist, d_ref, rtol=1e-6)
