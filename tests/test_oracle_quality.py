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
