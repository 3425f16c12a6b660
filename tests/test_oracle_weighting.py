"""Pins of the oracle's neighbourhood weighting: Eq. 1 (rho, sigma, membership)
and Eq. 2 (fuzzy union, read as the probabilistic t-conorm A + A^T - A o A^T).
"""

import json
import math
import os

import numpy as np
import pytest

from paper_2008_00325_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_sigma_closed_form(orc):
    g = _golden("smooth_knn_closed_form.json")
    d = np.array([g["distances"]], dtype=np.float32)
    rho, sigma = orc.smooth_knn(d)
    assert rho[0] == g["rho"]
    assert abs(sigma[0] - g["sigma"]) < 1e-5
    k = d.shape[1]
    # the closed form itself: 1 + (k-1) exp(-1/sigma) = log2 k
    assert abs(1 + (k - 1) * math.exp(-1 / g["sigma"]) - math.log2(k)) < 1e-5


def test_rho_is_smallest_positive_distance(orc):
    d = np.array([[0.0, 0.0, 0.7, 0.9, 3.0], [2.0, 1.5, 4.0, 5.0, 6.0], [0.0] * 5], dtype=np.float32)
    rho, sigma = orc.smooth_knn(d)
    assert rho[0] == np.float32(0.7) and rho[1] == np.float32(1.5) and rho[2] == 0.0
    # all-zero row: sigma floored at 1e-3 of the global mean distance
    assert sigma[2] >= 1e-3 * d.astype(np.float64).mean() - 1e-15


@pytest.mark.parametrize("k", [5, 15, 30])
def test_membership_sum_is_log2k(orc, k):
    bounds = synth.cluster_bounds(4000, 4)
    ids, dist = synth.window_knn(4000, k, bounds, seed=21)
    rho, sigma = orc.smooth_knn(dist)
    A = orc.membership(dist, rho, sigma)
    s = A.sum(axis=1)
    assert np.abs(s - math.log2(k)).max() < 1e-5
    # the nearest neighbour (distance rho) has membership exactly 1
    nearest = np.argmin(dist, axis=1)
    assert np.all(A[np.arange(4000), nearest] == 1.0)
    assert np.all((A > 0) & (A <= 1))


def test_sigma_against_brute_force_grid(orc):
    rng = np.random.default_rng(5)
    d = np.sort(rng.exponential(1.0, size=(40, 8)).cumsum(axis=1), axis=1).astype(np.float32)
    rho, sigma = orc.smooth_knn(d)
    grid = np.exp(np.linspace(np.log(1e-3), np.log(1e3), 200_001))
    target = math.log2(8)
    for i in range(d.shape[0]):
        x = np.maximum(d[i].astype(np.float64) - rho[i], 0.0)
        f = np.exp(-x[None, :] / grid[:, None]).sum(axis=1)
        best = grid[np.argmin(np.abs(f - target))]
        assert abs(sigma[i] / best - 1) < 1e-4


def test_union_toy_values(orc):
    g = _golden("fuzzy_union_toy.json")
    for case in g["cases"]:
        ids = np.array(case["ids"], dtype=np.int32)
        A = np.array(case["A"], dtype=np.float64)
        r, c, v = orc.fuzzy_union(ids, A)
        got = {(int(a), int(b)): float(x) for a, b, x in zip(r, c, v)}
        want = {(int(a), int(b)): float(x) for a, b, x in case["B"]}
        assert got.keys() == want.keys()
        for key in want:
            assert abs(got[key] - want[key]) < 1e-15


def test_union_properties_on_knn_graph(orc):
    X, _ = synth.blobs(300, 8, 3, seed=9)
    ids, dist = orc.exact_knn(X, 10)
    rho, sigma = orc.smooth_knn(dist)
    A = orc.membership(dist, rho, sigma)
    r, c, v = orc.fuzzy_union(ids, A)
    n = X.shape[0]
    Bd = {}
    for a, b, x in zip(r, c, v):
        Bd[(a, b)] = x
    Ad = {(i, int(ids[i, t])): A[i, t] for i in range(n) for t in range(ids.shape[1])}
    # bit-exact symmetry, and max(A_ij, A_ji) <= B_ij <= 1
    for (a, b), x in Bd.items():
        assert Bd[(b, a)] == x
        lo = max(Ad.get((a, b), 0.0), Ad.get((b, a), 0.0))
        assert lo - 1e-15 <= x <= 1.0
    mutual = sum(1 for (a, b) in Ad if (b, a) in Ad)
    assert len(Bd) == 2 * len(Ad) - mutual
    # sorted by (row, col)
    key = r.astype(np.int64) * n + c
    assert np.all(np.diff(key) > 0)


def test_union_rejects_duplicate_neighbours(orc):
    ids = np.array([[1, 1], [0, 2], [0, 1]], dtype=np.int32)
    with pytest.raises(ValueError):
        orc.fuzzy_union(ids, np.full((3, 2), 0.5))
