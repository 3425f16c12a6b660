"""Property tests of the oracle on random small inputs (hypothesis): the
invariants that Eq. 1, Eq. 2, the schedule, the ingest and the layout epoch
must satisfy for any input, not only for the fixed cases of the other pins."""

import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle as O

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@st.composite
def knn_lists(draw, max_n=40):
    """Random kNN lists: n vertices, k distinct neighbours each (self excluded),
    strictly increasing positive distances."""
    n = draw(st.integers(4, max_n))
    k = draw(st.integers(2, min(8, n - 1)))
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    ids = np.empty((n, k), dtype=np.int32)
    for i in range(n):
        others = np.delete(np.arange(n), i)
        ids[i] = rng.choice(others, size=k, replace=False)
    gaps = rng.uniform(0.01, 2.0, size=(n, k))
    dist = np.cumsum(gaps, axis=1).astype(np.float32)
    return ids, dist


@SETTINGS
@given(knn_lists())
def test_membership_sum_and_range(data):
    ids, dist = data
    k = ids.shape[1]
    rho, sigma = O.smooth_knn(dist)
    A = O.membership(dist, rho, sigma)
    total = A.sum(axis=1)
    # sigma is floored at 1e-3 x the row's mean distance (every rho > 0 here);
    # a row whose bisection would go below the floor keeps a sum above log2 k
    floor = 1e-3 * dist.astype(np.float64).mean(axis=1)
    free = sigma > floor * (1 + 1e-9)
    assert np.abs(total[free] - math.log2(k)).max(initial=0.0) < 1e-5
    assert np.all(total[~free] >= math.log2(k) - 1e-5)
    assert np.all(sigma >= floor * (1 - 1e-12))
    assert np.all((A > 0) & (A <= 1))
    assert np.all(A[:, 0] == 1.0)            # the nearest neighbour sits at rho
    assert np.all(np.asarray(rho, np.float32) == dist[:, 0])


@SETTINGS
@given(knn_lists())
def test_union_is_a_symmetric_t_conorm(data):
    ids, dist = data
    n, k = ids.shape
    rho, sigma = O.smooth_knn(dist)
    A = O.membership(dist, rho, sigma)
    r, c, v = O.fuzzy_union(ids, A)
    B = {(int(a), int(b)): float(x) for a, b, x in zip(r, c, v)}
    Ad = {}
    for i in range(n):
        for s in range(k):
            Ad[(i, int(ids[i, s]))] = float(A[i, s])
    # structure: the union of the directed entries and their transposes
    assert set(B) == set(Ad) | {(j, i) for (i, j) in Ad}
    for (i, j), b in B.items():
        assert B[(j, i)] == b                                 # bit-equal symmetry
        a, at = Ad.get((i, j), 0.0), Ad.get((j, i), 0.0)
        assert abs(b - (a + at - a * at)) <= 1e-12
        assert max(a, at) - 1e-12 <= b <= 1.0 + 1e-12
    # rows sorted by (row, col)
    key = r.astype(np.int64) * n + c
    assert np.all(np.diff(key) > 0)


@SETTINGS
@given(st.integers(1, 400), st.lists(st.floats(float(np.float32(1e-3)), 1.0, width=32), min_size=1, max_size=200))
def test_schedule_counts(N, ws):
    """Every kept edge is sampled exactly floor(N / eps) times, at most once an epoch."""
    v = np.float32(ws)
    w_max = v.max()
    v = v[v >= w_max / np.float32(N)]
    eps = (w_max / v).astype(np.float32)
    counts = np.zeros(eps.size, dtype=np.int64)
    for ep in range(N):
        counts += O.active_mask(eps, ep)
    assert np.array_equal(counts, np.floor(np.float32(N) / eps).astype(np.int64))


@SETTINGS
@given(knn_lists(max_n=30), st.integers(1, 60))
def test_prep_orders_and_prunes(data, N):
    ids, dist = data
    n = ids.shape[0]
    r, c, v = O.fuzzy_graph(ids, dist)
    g = O.prep(n, r, c, v, N)
    w_max = np.float32(v.max())
    keep = v >= w_max / np.float32(N)
    assert g.nnz == int(keep.sum())
    assert g.row_ptr[0] == 0 and g.row_ptr[-1] == g.nnz and np.all(np.diff(g.row_ptr) >= 0)
    heads = g.heads()
    key = heads.astype(np.int64) * n + g.col
    assert np.all(np.diff(key) > 0)
    kept = {(int(a), int(b)): np.float32(x) for a, b, x, k_ in zip(r, c, v, keep) if k_}
    for e in range(g.nnz):
        assert g.eps[e] == np.float32(w_max / kept[(int(heads[e]), int(g.col[e]))])


@SETTINGS
@given(knn_lists(max_n=30), st.integers(0, 6), st.integers(0, 2**32 - 1), st.integers(2, 50))
def test_pull_form_equals_push_form(data, R, seed, N):
    """The C oracle's push form (both endpoints per edge) and the numpy pull
    form (each row with twice its own share) give the same epoch."""
    ids, dist = data
    n = ids.shape[0]
    r, c, v = O.fuzzy_graph(ids, dist)
    g = O.prep(n, r, c, v, N)
    a, b = O.fit_ab(1.0, 0.1)
    E = np.random.default_rng(seed % (2**31)).uniform(-3, 3, size=(n, 2))
    for ep in sorted({0, N // 2, N - 1}):
        push, act = O.epoch(g, E, ep, a, b, N, R, seed)
        pull, act2 = O.frozen_epoch(g, E, E, ep, a, b, N, R, seed, attr_mult=2.0, self_skip=True)
        assert act == act2
        assert np.abs(push - pull).max() <= 1e-12 * max(1.0, np.abs(push).max())
