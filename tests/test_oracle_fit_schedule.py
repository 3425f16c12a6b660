"""Pins of the oracle's a/b fit (Eq. 3 target, smooth Phi) and of the ingest of
B with its edge schedule (sparse-data handling section; epochs-per-sample)."""

import json
import os

import numpy as np
import pytest
from scipy.optimize import curve_fit

from paper_2008_00325_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_ab_default_values(orc):
    g = json.load(open(os.path.join(GOLDEN, "ab_fit.json")))
    a, b = orc.fit_ab(g["spread"], g["min_dist"])
    assert abs(a - g["a"]) < 1e-3 and abs(b - g["b"]) < 1e-3


@pytest.mark.parametrize("spread,min_dist", [(1.0, 0.1), (1.0, 0.5), (2.0, 0.05), (0.5, 0.0)])
def test_ab_against_library_least_squares(orc, spread, min_dist):
    x = np.linspace(0.0, 3.0 * spread, 300)
    y = np.where(x < min_dist, 1.0, np.exp(-(x - min_dist) / spread))
    (ra, rb), _ = curve_fit(lambda x, a, b: 1.0 / (1.0 + a * x ** (2 * b)), x, y, p0=(1.0, 1.0), maxfev=20000)
    a, b = orc.fit_ab(spread, min_dist)
    assert abs(a - ra) < 2e-5 * max(1.0, abs(ra)) and abs(b - rb) < 2e-5


def _reference_prep(n, rows, cols, vals, n_epochs):
    """Independent numpy statement of the ingest (library sort, fp32 math)."""
    keep0 = (vals > 0) & (rows != cols)
    w_max = np.float32(vals[keep0].max()) if keep0.any() else np.float32(0)
    keep = keep0 & (vals >= w_max / np.float32(n_epochs))
    r, c, v = rows[keep], cols[keep], vals[keep]
    order = np.lexsort((c, r))
    r, c, v = r[order], c[order], v[order]
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    np.add.at(row_ptr, r + 1, 1)
    return np.cumsum(row_ptr), c, (w_max / v).astype(np.float32), w_max


def test_prep_matches_library_sort(orc):
    rows, cols, vals = synth.random_symmetric_coo(3000, 12, seed=4)
    # add zero entries, negative entries and self loops, which must be dropped
    rows = np.concatenate([rows, [5, 7, 9, 9]]).astype(np.int32)
    cols = np.concatenate([cols, [5, 8, 9, 10]]).astype(np.int32)
    vals = np.concatenate([vals, [0.9, 0.0, 0.5, -1.0]]).astype(np.float32)
    g = orc.prep(3000, rows, cols, vals, 200)
    rp, c, eps, w = _reference_prep(3000, rows, cols, vals, 200)
    assert g.w_max == w
    assert np.array_equal(g.row_ptr, rp)
    assert np.array_equal(g.col, c)
    assert np.array_equal(g.eps, eps)
    assert g.eps.min() == np.float32(1.0)


def test_prune_threshold_boundary(orc):
    # w_max = 1, N = 4: 0.25 is kept (sampled exactly once), the next float below is pruned
    below = np.nextafter(np.float32(0.25), np.float32(0))
    rows = np.array([0, 1, 0, 2, 0, 3], dtype=np.int32)
    cols = np.array([1, 0, 2, 0, 3, 0], dtype=np.int32)
    vals = np.array([1.0, 1.0, 0.25, 0.25, below, below], dtype=np.float32)
    g = orc.prep(4, rows, cols, vals, 4)
    assert g.nnz == 4
    assert list(g.col) == [1, 2, 0, 0]
    assert list(g.eps) == [1.0, 4.0, 1.0, 4.0]


def test_sample_count_closed_form(orc):
    """Edge e is active in exactly floor(N / eps_e) of the N epochs."""
    rng = np.random.default_rng(2)
    N = 200
    vals = np.concatenate([rng.random(20000).astype(np.float32), np.float32([1.0, 0.5, 0.25, 1 / 3, 0.005, 0.01])])
    vals = vals[vals >= np.float32(1.0) / np.float32(N)]
    eps = (np.float32(1.0) / vals).astype(np.float32)
    counts = np.zeros(eps.size, dtype=np.int64)
    for ep in range(N):
        counts += orc.active_mask(eps, ep)
    assert np.array_equal(counts, np.floor(np.float32(N) / eps).astype(np.int64))
    # eps = 1 edges are active in every epoch, including epoch 0
    assert orc.active(1.0, 0) and orc.active(1.0, N - 1)
    assert orc.active_mask(np.float32([3.0]), 0)[0] == False  # noqa: E712
    assert orc.active_mask(np.float32([3.0]), 2)[0] == True  # noqa: E712
    # the scalar C predicate and the vectorised one agree
    for t in range(0, eps.size, 997):
        for ep in (0, 1, 57, N - 1):
            assert orc.active(float(eps[t]), ep) == bool(orc.active_mask(eps[t:t + 1], ep)[0])


def test_prep_errors(orc):
    r = np.array([0, 1], dtype=np.int32)
    c = np.array([1, 0], dtype=np.int32)
    v = np.array([0.5, 0.5], dtype=np.float32)
    with pytest.raises(orc.PrepError) as ei:
        orc.prep(2, r, c, np.array([0.5, 0.25], dtype=np.float32), 10)
    assert ei.value.status == -2
    with pytest.raises(orc.PrepError) as ei:
        orc.prep(2, np.array([0], dtype=np.int32), np.array([1], dtype=np.int32), np.float32([0.5]), 10)
    assert ei.value.status == -2
    with pytest.raises(orc.PrepError) as ei:
        orc.prep(2, np.array([0, 1, 0], dtype=np.int32), np.array([1, 0, 1], dtype=np.int32),
                 np.float32([0.5, 0.5, 0.5]), 10)
    assert ei.value.status == -1
    with pytest.raises(orc.PrepError) as ei:
        orc.prep(2, r, np.array([1, 2], dtype=np.int32), v, 10)
    assert ei.value.status == -1
    with pytest.raises(orc.PrepError) as ei:
        orc.prep(2, r, c, np.float32([np.nan, 0.5]), 10)
    assert ei.value.status == -1
    # empty and all-dropped inputs are valid and keep nothing
    g = orc.prep(3, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), 10)
    assert g.nnz == 0 and np.all(g.row_ptr == 0)
    g = orc.prep(3, np.array([1], np.int32), np.array([1], np.int32), np.float32([1.0]), 10)
    assert g.nnz == 0
