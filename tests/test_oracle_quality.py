"""Pins of the oracle's evaluation helpers: exact kNN (kNN-graph section) and
trustworthiness (Alg. 1, with the Venna-Kaski normalisation the experiments
section cites), against scikit-learn's independent implementations."""

import numpy as np
from sklearn.manifold import trustworthiness as sk_trust
from sklearn.neighbors import NearestNeighbors

from paper_2008_00325_amd import synth


def test_exact_knn_matches_library(orc):
    X, _ = synth.blobs(600, 16, 5, seed=3)
    ids, dist = orc.exact_knn(X, 15, batch=128)
    nn = NearestNeighbors(n_neighbors=16, algorithm="brute").fit(X.astype(np.float64))
    d_ref, i_ref = nn.kneighbors(X.astype(np.float64))
    assert np.array_equal(np.sort(ids, axis=1), np.sort(i_ref[:, 1:], axis=1))
    assert np.allclose(dist, d_ref[:, 1:], rtol=1e-6)
    assert np.all(np.diff(dist, axis=1) >= 0)
    assert not np.any(ids == np.arange(600)[:, None])


def test_trustworthiness_matches_library(orc):
    X, _ = synth.blobs(400, 12, 4, seed=8)
    rng = np.random.default_rng(1)
    for Y in (X[:, :2], rng.normal(size=(400, 2)), X[:, :3] + 0.3 * rng.normal(size=(400, 3))):
        for k in (5, 15):
            assert abs(orc.trustworthiness(X, Y, k) - sk_trust(X, Y, n_neighbors=k)) < 1e-9


def test_trustworthiness_identity_and_sampled_rows(orc):
    X, _ = synth.blobs(300, 6, 3, seed=2)
    assert orc.trustworthiness(X, X, 10) == 1.0
    Y = X[:, :2]
    full = orc.trustworthiness(X, Y, 10)
    # the row-sampled form over all rows is the full sum
    assert abs(orc.trustworthiness(X, Y, 10, rows=np.arange(300)) - full) < 1e-12


# ---------------------------------------------------------------------------
# recall@k and the objective (graph-only workloads)
# ---------------------------------------------------------------------------

def test_recall_of_exact_knn_is_one(orc):
    """The input lists are the exact kNN of the layout itself (brute force):
    every neighbour is found again by the k-d tree."""
    rng = np.random.default_rng(4)
    Y = rng.normal(size=(3000, 2))
    ids, _ = orc.exact_knn(Y, 15, batch=512)
    rows = np.arange(0, 3000, 7)
    assert orc.recall_at_k(ids, Y, rows, 15) == 1.0
    assert orc.recall_at_k(ids, Y, rows, 5) == 1.0
    # a layout unrelated to the lists finds almost none of them
    Z = rng.normal(size=(3000, 2))
    assert orc.recall_at_k(ids, Z, rows, 15) < 0.02


def test_recall_by_hand_on_a_line():
    """Points at 0, 1, 3, 6, 10, ... (gaps 1, 2, 3, ...): the nearest other
    point of i is i - 1 (i >= 1) and 1 for i = 0.  With each list naming i + 1
    first (n - 2 for the last point), recall@1 = 2 / n."""
    import oracle as O

    n = 12
    Y = np.cumsum(np.arange(n))[:, None].astype(np.float64)
    ids = np.array([[i + 1] if i < n - 1 else [n - 2] for i in range(n)])
    assert abs(O.recall_at_k(ids, Y, np.arange(n), 1) - 2.0 / n) < 1e-15


def _pair_graph(orc):
    return orc.prep(2, np.array([0, 1], np.int32), np.array([1, 0], np.int32), np.array([1.0, 1.0], np.float32), 10)


def test_objective_two_points_closed_form(orc):
    """Two points joined both ways with weight 1 (sampled every epoch), a = b = 1:
    at distance 1, Phi = 1/2, so every attraction and every repulsion term is
    ln 2; at distance 2, Phi = 1/5: the terms are ln 5 and ln(5/4)."""
    g = _pair_graph(orc)
    rows = np.array([0, 1])
    neg = np.array([[1, 1, 1], [0, 0, 0]])
    R = 5
    Y1 = np.array([[0.0, 0.0], [1.0, 0.0]])
    assert abs(orc.objective(g, Y1, 1.0, 1.0, R, rows, neg) - 12.0 * np.log(2.0)) < 1e-12
    Y2 = np.array([[0.0, 0.0], [0.0, 2.0]])
    assert abs(orc.objective(g, Y2, 1.0, 1.0, R, rows, neg) - 2.0 * (np.log(5.0) + R * np.log(1.25))) < 1e-12
    # a negative equal to its source is skipped, not counted in the mean
    neg_self = np.array([[0, 1, 0], [1, 0, 1]])
    assert abs(orc.objective(g, Y1, 1.0, 1.0, R, rows, neg_self) - 12.0 * np.log(2.0)) < 1e-12
    # only the sampled rows count
    assert abs(orc.objective(g, Y1, 1.0, 1.0, R, rows[:1], neg[:1]) - 6.0 * np.log(2.0)) < 1e-12


def test_objective_derivative_is_the_attraction(orc):
    """Without negatives the objective of row 0 is -log Phi(y_0, y_1); its
    derivative in y_0 is minus the attraction (pinned above by finite
    differences of log Phi)."""
    g = _pair_graph(orc)
    a, b = 1.577, 0.895
    rng = np.random.default_rng(2)
    for _ in range(20):
        Y = rng.normal(size=(2, 2)) * 2
        h = 1e-6
        fd = []
        for e in np.eye(2):
            Yp, Ym = Y.copy(), Y.copy()
            Yp[0] += h * e
            Ym[0] -= h * e
            fd.append((orc.objective(g, Yp, a, b, 0, np.array([0]), np.zeros((1, 0), np.int64))
                       - orc.objective(g, Ym, a, b, 0, np.array([0]), np.zeros((1, 0), np.int64))) / (2 * h))
        diff = Y[0] - Y[1]
        assert np.allclose(fd, -orc.attr_coef(float(diff @ diff), a, b) * diff, rtol=1e-6, atol=1e-8)
