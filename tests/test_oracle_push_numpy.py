"""Pins of the oracle against independent writings from the paper's text.

* The epoch: a literal push-form Jacobi epoch written here in plain Python
  (no code shared with the C oracle: its own Philox4x32-10 from Salmon et al.,
  SC'11, its own fp32 schedule test, its own gradient terms), run on random
  small graphs, must equal the C oracle's epoch.  "Push form" is the
  embedding-updates section read literally: a sampled edge (i, j) moves y_i by
  +alpha g and y_j by -alpha g, and each of its neg_rate draws k moves y_i
  alone; every term is computed from the snapshot E_n and applied at the end
  of the epoch (the deterministic mode of the reproducibility section).
* The kNN tie rule: exact_knn orders neighbours by (distance, index), checked
  by brute force on inputs made of ties (a line of integers, a lattice,
  repeated points).
"""

import math

import numpy as np
import pytest

import oracle as O
from paper_2008_00325_amd import synth

M32 = 0xFFFFFFFF


def philox_block(ctr, key):
    """Philox4x32-10 on one counter (four 32-bit words), key (two words):
    ten rounds of two 32x32->64 products by 0xD2511F53 and 0xCD9E8D57, whose
    high halves are xored with the other two words and the round key; the
    key is bumped by 0x9E3779B9 and 0xBB67AE85 after each round."""
    c0, c1, c2, c3 = ctr
    k0, k1 = key
    for _ in range(10):
        p0 = 0xD2511F53 * c0
        p1 = 0xCD9E8D57 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0) & M32, p1 & M32, ((p0 >> 32) ^ c3 ^ k1) & M32, p0 & M32
        k0 = (k0 + 0x9E3779B9) & M32
        k1 = (k1 + 0xBB67AE85) & M32
    return c0, c1, c2, c3


def negative_vertex(seed, epoch, e, r, n):
    """Draw r of edge e in `epoch` (reading C17): word r & 3 of the counter
    (lo32 e, hi32 e, epoch, 0x4E470000 | r >> 2), mapped to [0, n) by the
    high half of word * n."""
    words = philox_block((e & M32, e >> 32, epoch, 0x4E470000 | (r >> 2)), (seed & M32, seed >> 32))
    return (words[r & 3] * n) >> 32


def sampled(eps, epoch):
    """Reading C10 in fp32: floor((n + 1) / eps) > floor(n / eps)."""
    f = np.float32
    return bool(np.floor(f(epoch + 1) / f(eps)) > np.floor(f(epoch) / f(eps)))


def clip(x):
    return min(4.0, max(-4.0, x))


def push_epoch(n, dim, row_ptr, col, eps, E, epoch, a, b, n_epochs, neg_rate, seed):
    alpha = 1.0 - epoch / n_epochs
    D = [[0.0] * dim for _ in range(n)]
    Y = [[float(x) for x in row] for row in E]
    active = 0
    for i in range(n):
        for e in range(int(row_ptr[i]), int(row_ptr[i + 1])):
            if not sampled(eps[e], epoch):
                continue
            active += 1
            j = int(col[e])
            diff = [Y[i][d] - Y[j][d] for d in range(dim)]
            d2 = sum(x * x for x in diff)
            # d/dy_i log Phi, Phi = 1 / (1 + a d^(2b)): -2ab d^(2(b-1)) / (1 + a d^(2b)) (0 at d = 0)
            c = -2.0 * a * b * d2 ** (b - 1.0) / (1.0 + a * d2 ** b) if d2 > 0.0 else 0.0
            for d in range(dim):
                g = clip(c * diff[d])
                D[i][d] += alpha * g          # the source ...
                D[j][d] -= alpha * g          # ... and the other endpoint
            for r in range(neg_rate):
                k = negative_vertex(seed, epoch, e, r, n)
                if k == i:
                    continue
                diff = [Y[i][d] - Y[k][d] for d in range(dim)]
                d2 = sum(x * x for x in diff)
                # d/dy_i log(1 - Phi) with gamma = 1, (1e-3 + d^2): 2b / ((1e-3 + d2)(1 + a d2^b))
                c = 2.0 * b / ((1e-3 + d2) * (1.0 + a * d2 ** b)) if d2 > 0.0 else 0.0
                for d in range(dim):
                    D[i][d] += alpha * clip(c * diff[d])   # the source only
    out = np.array([[Y[i][d] + D[i][d] for d in range(dim)] for i in range(n)])
    return out, active


@pytest.mark.parametrize("n,deg,dim,R,N,seed", [
    (12, 3, 2, 0, 10, 1), (12, 3, 2, 5, 10, 2), (30, 6, 2, 5, 40, 3), (50, 8, 3, 5, 200, 4),
    (50, 4, 1, 0, 7, 5), (41, 10, 2, 5, 3, 2**40 + 17),
])
def test_c_oracle_epoch_equals_plain_push_form(n, deg, dim, R, N, seed):
    r, c, v = synth.random_symmetric_coo(n, deg, seed=n * 7 + deg)
    g = O.prep(n, r, c, v, N)
    a, b = O.fit_ab(1.0, 0.1)
    E = np.random.default_rng(seed % 1000).uniform(-4.0, 4.0, size=(n, dim))
    for ep in sorted({0, N // 2, N - 1}):
        want, act = push_epoch(n, dim, g.row_ptr, g.col, g.eps, E, ep, a, b, N, R, seed)
        got, act_c = O.epoch(g, E, ep, a, b, N, R, seed)
        assert act == act_c
        assert np.abs(got - want).max() <= 1e-12 * max(1.0, np.abs(want).max())


def test_plain_philox_matches_the_oracle_draws():
    """The two writings of the negative stream agree (the oracle's is pinned
    to an independent C++ implementation elsewhere)."""
    seed, n = 0x1234_5678_9ABC_DEF0, 1_000_003
    got = O.negative_vertices(seed, 7, 100, 50, 6, n)
    for t in range(50):
        for r in range(6):
            assert got[t, r] == negative_vertex(seed, 7, 100 + t, r, n)


def test_push_form_moves_both_endpoints_by_hand():
    """Two points 1 apart on a line, one edge pair, no negatives, a = b = 1:
    c = -2 / (1 + 1) = -1, g = clip(-1 * (y0 - y1)) = 1 for y0 - y1 = -1, so
    in epoch 0 (alpha = 1) each of the two directed edges moves its source by
    +-1 toward the other and its other endpoint by the opposite: y0 gains
    1 (own edge) + 1 (as the other endpoint of (1, 0)) and the points swap."""
    row_ptr = np.array([0, 1, 2])
    col = np.array([1, 0])
    eps = np.float32([1.0, 1.0])
    out, act = push_epoch(2, 1, row_ptr, col, eps, np.array([[0.0], [1.0]]), 0, 1.0, 1.0, 10, 0, 0)
    assert act == 2
    assert out.tolist() == [[2.0], [-1.0]]


def _brute_knn(X, k):
    X = X.astype(np.float64)
    n = X.shape[0]
    ids = np.empty((n, k), dtype=np.int64)
    for i in range(n):
        d = np.sqrt(((X - X[i]) ** 2).sum(1))
        order = sorted((j for j in range(n) if j != i), key=lambda j: (d[j], j))
        ids[i] = order[:k]
    return ids


@pytest.mark.parametrize("kind,k", [("line", 5), ("lattice", 8), ("repeats", 12), ("repeats", 29)])
def test_exact_knn_orders_ties_by_index(kind, k):
    if kind == "line":
        X = np.arange(40, dtype=np.float32)[:, None]
    elif kind == "lattice":
        X = np.stack(np.meshgrid(np.arange(7), np.arange(6)), -1).reshape(-1, 2).astype(np.float32)
    else:
        X = np.zeros((30, 3), np.float32)
        X[10:] = 1.0
        X[20:] = np.float32([1.0, 2.0, 3.0])
    ids, dist = O.exact_knn(X, k, batch=7)
    assert np.array_equal(ids, _brute_knn(X, k))
    want = np.sqrt(((X[ids].astype(np.float64) - X[:, None, :].astype(np.float64)) ** 2).sum(-1))
    assert np.array_equal(dist, want.astype(np.float32))
    assert math.isfinite(float(dist.max()))
