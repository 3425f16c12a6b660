"""CPU oracle for the UMAP layout path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  The product library never loads it, and it shares
no code with the GPU path.  The arithmetic lives in ``umap_oracle.c`` (fp64
state, fp32 schedule); this module marshals numpy arrays into it and adds two
plain numpy routines (exact kNN and trustworthiness).

Paper: Nolet et al., "Bringing UMAP Closer to the Speed of Light with GPU
Acceleration" (AAAI 2021).  Each function cites the passage it follows.

Parity status of each function is recorded next to it: "pinned" functions are
checked by tests against closed forms, independent library routines or brute
force; none is unpinned.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "umap_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

GCC_CMD = ["gcc", "-std=c11", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", _LIB, _SRC, "-lm"]


def build() -> str:
    """Compile the oracle library with gcc (always recompiles)."""
    subprocess.run(GCC_CMD, check=True)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        i32, i64, u32, u64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_double
        P = ctypes.c_void_p
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_philox_batch.argtypes = [P, i64, P, P]
        L.orc_negative_vertex.argtypes = [u64, i64, i32, i32, i64]
        L.orc_negative_vertex.restype = u32
        L.orc_negative_batch.argtypes = [u64, i32, i64, i64, i32, i64, P]
        L.orc_init.argtypes = [i64, i32, u64, P]
        L.orc_smooth_knn.argtypes = [i64, i32, P, P, P]
        L.orc_membership.argtypes = [i64, i32, P, P, P, P]
        L.orc_fuzzy_union.argtypes = [i64, i32, P, P, P, P, P]
        L.orc_fuzzy_union.restype = i64
        L.orc_fit_ab.argtypes = [f64, f64, P, P]
        L.orc_active.argtypes = [ctypes.c_float, i32]
        L.orc_active.restype = ctypes.c_int
        L.orc_prep.argtypes = [i64, P, P, P, i64, i32, P, P, P, P]
        L.orc_prep.restype = i64
        L.orc_attr_coef.argtypes = [f64, f64, f64]
        L.orc_attr_coef.restype = f64
        L.orc_rep_coef.argtypes = [f64, f64, f64]
        L.orc_rep_coef.restype = f64
        L.orc_epoch.argtypes = [i64, i32, P, P, P, f64, f64, i32, i32, u64, i32, P, P]
        L.orc_epoch.restype = i64
        L.orc_epoch_rows.argtypes = [i64, i32, P, P, P, f64, f64, i32, i32, u64, i32, P, i64, P, P]
        L.orc_run.argtypes = [i64, i32, P, P, P, f64, f64, i32, i32, u64, P, P]
        L.orc_num_threads.restype = ctypes.c_int
        L.orc_set_num_threads.argtypes = [i32]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return int(lib().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's later parallel regions (results do not depend on it)."""
    lib().orc_set_num_threads(n)


# --------------------------------------------------------------------------
# Random streams (Philox4x32-10, SC'11).  Pinned against an independent
# implementation of the same generator and by uniformity tests.
# --------------------------------------------------------------------------

def philox4x32_10(counters: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    ctr = _c(counters, np.uint32).reshape(-1, 4)
    k = np.array(key, dtype=np.uint32)
    out = np.empty_like(ctr)
    lib().orc_philox_batch(_p(k), ctr.shape[0], _p(ctr), _p(out))
    return out


def negative_vertices(seed: int, epoch: int, e_first: int, count: int, neg_rate: int, n: int) -> np.ndarray:
    out = np.empty((count, neg_rate), dtype=np.uint32)
    lib().orc_negative_batch(seed, epoch, e_first, count, neg_rate, n, _p(out))
    return out


def init_layout(n: int, dim: int, seed: int) -> np.ndarray:
    """Random initial layout, uniform on [-10, 10) (embedding-updates section)."""
    out = np.empty((n, dim), dtype=np.float32)
    lib().orc_init(n, dim, seed, _p(out))
    return out


# --------------------------------------------------------------------------
# Neighbourhood weighting: Eq. 1 (smooth kNN) and Eq. 2 (fuzzy union).
# --------------------------------------------------------------------------

def smooth_knn(dists: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """rho and sigma per vertex (Eq. 1; neighbourhood-weighting section)."""
    d = _c(dists, np.float32)
    n, k = d.shape
    rho = np.empty(n)
    sigma = np.empty(n)
    lib().orc_smooth_knn(n, k, _p(d), _p(rho), _p(sigma))
    return rho, sigma


def membership(dists: np.ndarray, rho: np.ndarray, sigma: np.ndarray) -> np.ndarray:
    """A_ij = exp(-max(0, d_ij - rho_i) / sigma_i) (summand of Eq. 1)."""
    d = _c(dists, np.float32)
    n, k = d.shape
    A = np.empty((n, k))
    lib().orc_membership(n, k, _p(d), _p(_c(rho, np.float64)), _p(_c(sigma, np.float64)), _p(A))
    return A


def fuzzy_union(ids: np.ndarray, A: np.ndarray):
    """B = A + A^T - A o A^T as COO sorted by (row, col), fp64 values (Eq. 2,
    read with the t-conorm's minus sign)."""
    ids = _c(ids, np.int32)
    A = _c(A, np.float64)
    n, k = ids.shape
    cap = 2 * n * k
    rows = np.empty(cap, dtype=np.int32)
    cols = np.empty(cap, dtype=np.int32)
    vals = np.empty(cap, dtype=np.float64)
    m = lib().orc_fuzzy_union(n, k, _p(ids), _p(A), _p(rows), _p(cols), _p(vals))
    if m < 0:
        raise ValueError("invalid kNN lists (duplicate neighbour or id out of range)")
    return rows[:m].copy(), cols[:m].copy(), vals[:m].copy()


def fuzzy_graph(ids: np.ndarray, dists: np.ndarray):
    """kNN lists -> symmetric COO graph with fp32 values (the layout's input)."""
    rho, sigma = smooth_knn(dists)
    A = membership(dists, rho, sigma)
    r, c, v = fuzzy_union(ids, A)
    return r, c, v.astype(np.float32)


def fit_ab(spread: float = 1.0, min_dist: float = 0.1) -> tuple[float, float]:
    """(a, b) of 1/(1 + a x^(2b)) fitted to the target curve of Eq. 3."""
    a = ctypes.c_double()
    b = ctypes.c_double()
    lib().orc_fit_ab(spread, min_dist, ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


# --------------------------------------------------------------------------
# Edge schedule and the ingest of B.
# --------------------------------------------------------------------------

def active(eps: float, epoch: int) -> bool:
    return bool(lib().orc_active(np.float32(eps), epoch))


def active_mask(eps: np.ndarray, epoch: int) -> np.ndarray:
    """Vectorised predicate in fp32 (floor((n+1)/eps) > floor(n/eps))."""
    e = _c(eps, np.float32)
    now = np.floor(np.float32(epoch + 1) / e)
    before = np.floor(np.float32(epoch) / e)
    return now > before


class Graph:
    """Kept edges of B sorted by (head, tail) with a CSR index."""

    def __init__(self, n, row_ptr, col, eps, w_max):
        self.n = n
        self.row_ptr = row_ptr
        self.col = col
        self.eps = eps
        self.w_max = w_max

    @property
    def nnz(self) -> int:
        return int(self.col.size)

    def heads(self) -> np.ndarray:
        return np.repeat(np.arange(self.n, dtype=np.int32), np.diff(self.row_ptr))


class PrepError(ValueError):
    def __init__(self, status: int):
        super().__init__({-1: "invalid graph", -2: "asymmetric graph"}.get(status, str(status)))
        self.status = status


def prep(n: int, rows, cols, vals, n_epochs: int) -> Graph:
    """Drop/prune/sort/eps of the COO graph (sparse-data handling section)."""
    rows = _c(rows, np.int32)
    cols = _c(cols, np.int32)
    vals = _c(vals, np.float32)
    nnz = rows.size
    row_ptr = np.empty(n + 1, dtype=np.int64)
    col = np.empty(max(nnz, 1), dtype=np.int32)
    eps = np.empty(max(nnz, 1), dtype=np.float32)
    w = ctypes.c_float()
    kept = lib().orc_prep(n, _p(rows), _p(cols), _p(vals), nnz, n_epochs, _p(row_ptr), _p(col), _p(eps),
                          ctypes.byref(w))
    if kept < 0:
        raise PrepError(int(kept))
    return Graph(n, row_ptr, col[:kept].copy(), eps[:kept].copy(), w.value)


# --------------------------------------------------------------------------
# Layout SGD (objective of the UMAP section; embedding-updates and
# reproducibility sections).
# --------------------------------------------------------------------------

def attr_coef(d2: float, a: float, b: float) -> float:
    return lib().orc_attr_coef(d2, a, b)


def rep_coef(d2: float, a: float, b: float) -> float:
    return lib().orc_rep_coef(d2, a, b)


def epoch(g: Graph, E: np.ndarray, epoch_idx: int, a: float, b: float, n_epochs: int, neg_rate: int,
          seed: int) -> tuple[np.ndarray, int]:
    """One Jacobi epoch from snapshot E (fp64 push form).  Returns (E', active)."""
    E = _c(E, np.float64)
    n, dim = E.shape
    out = np.empty_like(E)
    act = lib().orc_epoch(n, dim, _p(g.row_ptr), _p(g.col), _p(g.eps), a, b, n_epochs, neg_rate, seed,
                          epoch_idx, _p(E), _p(out))
    return out, int(act)


def epoch_rows(g: Graph, E: np.ndarray, epoch_idx: int, a: float, b: float, n_epochs: int, neg_rate: int,
               seed: int, which: np.ndarray) -> np.ndarray:
    """Update landing on the vertices `which` in one epoch (push form)."""
    E = _c(E, np.float64)
    n, dim = E.shape
    which = _c(which, np.int64)
    delta = np.empty((which.size, dim))
    lib().orc_epoch_rows(n, dim, _p(g.row_ptr), _p(g.col), _p(g.eps), a, b, n_epochs, neg_rate, seed,
                         epoch_idx, _p(E), which.size, _p(which), _p(delta))
    return delta


def run(g: Graph, dim: int, a: float, b: float, n_epochs: int, neg_rate: int, seed: int):
    """Init + all epochs.  Returns (E_N fp64, active counts per epoch)."""
    E = np.empty((g.n, dim))
    act = np.empty(n_epochs, dtype=np.int64)
    rc = lib().orc_run(g.n, dim, _p(g.row_ptr), _p(g.col), _p(g.eps), a, b, n_epochs, neg_rate, seed,
                       _p(E), _p(act))
    if rc != 0:
        raise MemoryError("oracle run failed")
    return E, act


# --------------------------------------------------------------------------
# Plain numpy: exact kNN (kNN-graph section) and trustworthiness (Alg. 1;
# Venna and Kaski's definition, which the experiments section cites).
# --------------------------------------------------------------------------

def _sqdist(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    A = A.astype(np.float64)
    B = B.astype(np.float64)
    d = (A * A).sum(1)[:, None] + (B * B).sum(1)[None, :] - 2.0 * (A @ B.T)
    return np.maximum(d, 0.0)


def exact_knn(X: np.ndarray, k: int, batch: int = 1024) -> tuple[np.ndarray, np.ndarray]:
    """k nearest neighbours of every row (self excluded), Euclidean, ties by
    smaller index.  Distances are recomputed exactly in fp64 for the chosen ids."""
    X64 = X.astype(np.float64)
    n = X.shape[0]
    ids = np.empty((n, k), dtype=np.int32)
    dist = np.empty((n, k), dtype=np.float32)
    for s in range(0, n, batch):
        t = min(n, s + batch)
        D = _sqdist(X64[s:t], X64)
        D[np.arange(t - s), np.arange(s, t)] = np.inf
        # every point whose (rounded) squared distance is within a relative
        # 1e-9 of the k-th smallest is a candidate, so that no tie at the k-th
        # distance (nor a pair the rounding of D misorders) is cut off
        kth = np.partition(D, k - 1, axis=1)[:, k - 1]
        cut = kth * (1.0 + 1e-9) + 1e-300
        width = int((D <= cut[:, None]).sum(axis=1).max())
        cand = np.argpartition(D, width - 1, axis=1)[:, :width] if width < n else np.tile(np.arange(n), (t - s, 1))
        cd = np.take_along_axis(D, cand, axis=1)
        # exact fp64 distances of the candidates, then order by (distance, index)
        diff = X64[s:t, None, :] - X64[cand]
        ed = np.sqrt((diff * diff).sum(-1))
        ed[~np.isfinite(cd)] = np.inf
        order = np.lexsort((cand, ed), axis=1)[:, :k]
        ids[s:t] = np.take_along_axis(cand, order, axis=1)
        dist[s:t] = np.take_along_axis(ed, order, axis=1)
    return ids, dist


def trustworthiness(X: np.ndarray, Y: np.ndarray, k: int = 15, rows: np.ndarray | None = None,
                    batch: int = 256) -> float:
    """T(k) = 1 - 2/(n k (2n - 3k - 1)) * sum_i sum_{j in U_k(i)} (r(i, j) - k),
    where U_k(i) are the embedding's k nearest neighbours of i that are not
    among its k nearest input neighbours and r(i, j) is the 1-based rank of j
    by input distance from i (self excluded, ties by index).  With `rows`, the
    sum runs over those rows only and is rescaled by n / len(rows) (a sampled
    estimate, identical for any two embeddings compared on the same rows)."""
    n = X.shape[0]
    if rows is None:
        rows = np.arange(n)
    rows = np.asarray(rows, dtype=np.int64)
    X64 = X.astype(np.float64)
    Y64 = Y.astype(np.float64)
    total = 0.0
    for s in range(0, rows.size, batch):
        r = rows[s: s + batch]
        DX = _sqdist(X64[r], X64)
        DX[np.arange(r.size), r] = -np.inf          # self ranks first (rank 0)
        DY = _sqdist(Y64[r], Y64)
        DY[np.arange(r.size), r] = np.inf
        nn_y = np.argpartition(DY, k, axis=1)[:, :k]
        for t in range(r.size):
            order = np.lexsort((np.arange(n), DX[t]))
            rank = np.empty(n, dtype=np.int64)
            rank[order] = np.arange(n)
            rk = rank[nn_y[t]]
            total += float(np.maximum(rk - k, 0).sum())
    total *= n / rows.size
    return 1.0 - 2.0 / (n * k * (2.0 * n - 3.0 * k - 1.0)) * total


# --------------------------------------------------------------------------
# Quality of graph-only workloads (no input coordinates, so no
# trustworthiness): neighbour recall and the objective of the UMAP section on
# a seeded vertex sample.
# --------------------------------------------------------------------------

def recall_at_k(knn_ids: np.ndarray, Y: np.ndarray, rows: np.ndarray, k: int = 15) -> float:
    """Mean over `rows` of |N_in(i) & N_emb(i)| / k, N_in(i) the first k
    entries of i's input neighbour list (nearest first), N_emb(i) the k
    nearest other vertices of i in the layout Y (Euclidean in fp64; a k-d tree
    finds them, ties in any order).  Pinned: 1 for the exact kNN of Y itself;
    hand-checked counts on a small line layout."""
    from scipy.spatial import cKDTree

    Y64 = np.asarray(Y, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    _, nb = cKDTree(Y64).query(Y64[rows], k=k + 1)
    hits = 0
    for t, i in enumerate(rows):
        emb = [int(j) for j in nb[t] if j != i][:k]
        hits += len(set(emb) & set(int(j) for j in knn_ids[i, :k]))
    return hits / (k * rows.size)


def objective(g: Graph, Y: np.ndarray, a: float, b: float, neg_rate: int, rows: np.ndarray,
              negatives: np.ndarray) -> float:
    """The cross-entropy objective of the UMAP section, restricted to the edges
    of the sampled vertices `rows`:
        sum_i sum_{e = (i, j)} f_e ( -log Phi(y_i, y_j)
                                      - neg_rate * mean_c log(1 - Phi(y_i, y_c)) ),
    Phi(x, y) = 1 / (1 + a |x - y|^(2b)), f_e = 1 / eps_e the fraction of epochs
    in which e is sampled, c over the fixed vertices negatives[t] of the t-th
    row (c = i skipped).  log(1 - Phi) is taken as log(a d^(2b) / (1 + a d^(2b)))
    with d^2 floored at 1e-12 (coincident points).  Pinned: closed-form values
    on two points; its derivative matches the gradient coefficients."""
    Y64 = np.asarray(Y, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    total = 0.0
    for t, i in enumerate(rows):
        lo, hi = int(g.row_ptr[i]), int(g.row_ptr[i + 1])
        if hi == lo:
            continue
        f = 1.0 / g.eps[lo:hi].astype(np.float64)
        d2 = ((Y64[g.col[lo:hi]] - Y64[i]) ** 2).sum(1)
        attract = np.log1p(a * d2 ** b)                       # -log Phi
        c = negatives[t][negatives[t] != i]
        dc2 = np.maximum(((Y64[c] - Y64[i]) ** 2).sum(1), 1e-12)
        p = a * dc2 ** b
        repel = -(np.log(p) - np.log1p(p)).mean() if c.size else 0.0   # -log(1 - Phi)
        total += float((f * (attract + neg_rate * repel)).sum())
    return total


# --------------------------------------------------------------------------
# Transform (inference): new points laid out against a frozen trained layout;
# only the new points move (embedding-updates section; model section on the
# kept kNN index).  Plain numpy, fp64 state, the fp32 schedule of `prep`.
# --------------------------------------------------------------------------

def prep_bipartite(n: int, n_table: int, rows, cols, vals, n_epochs: int) -> Graph:
    """Drop/prune/sort/eps of the graph from n new points (rows) to the n_table
    vertices of a frozen layout (columns): the steps of `prep` without the
    self-loop drop (a row and a column with the same index are different
    vertices) and without the symmetry requirement."""
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    vals = np.asarray(vals, dtype=np.float32)
    if rows.size and (rows.min() < 0 or rows.max() >= n or cols.min() < 0 or cols.max() >= n_table):
        raise PrepError(-1)
    if not np.all(np.isfinite(vals)):
        raise PrepError(-1)
    cand = vals > 0
    w_max = np.float32(vals[cand].max()) if cand.any() else np.float32(0)
    keep = cand & (vals >= w_max / np.float32(n_epochs))
    r, c, v = rows[keep], cols[keep], vals[keep]
    order = np.lexsort((c, r))
    r, c, v = r[order], c[order], v[order]
    if r.size > 1 and np.any((r[1:] == r[:-1]) & (c[1:] == c[:-1])):
        raise PrepError(-1)
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(np.bincount(r, minlength=n))
    eps = (w_max / v).astype(np.float32)
    return Graph(n, row_ptr, c.astype(np.int32), eps, float(w_max))


def transform_init(g: Graph, T: np.ndarray) -> np.ndarray:
    """Initial position of each new point: the mean of its kept neighbours'
    positions in the frozen layout T, weighted by 1/eps_e (the edge weight over
    w_max); a point without kept edges starts at the origin."""
    T64 = np.asarray(T, dtype=np.float64)
    w = 1.0 / g.eps.astype(np.float64)
    heads = g.heads()
    num = np.zeros((g.n, T64.shape[1]))
    den = np.zeros(g.n)
    np.add.at(num, heads, w[:, None] * T64[g.col])
    np.add.at(den, heads, w)
    Y = np.zeros_like(num)
    has = den > 0
    Y[has] = num[has] / den[has, None]
    return Y


def _attr_coef_v(d2: np.ndarray, a: float, b: float) -> np.ndarray:
    """d/dy_i log Phi = c (y_i - y_j), c = -2ab d2^(b-1) / (1 + a d2^b); 0 at d2 = 0."""
    safe = np.where(d2 > 0, d2, 1.0)
    return np.where(d2 > 0, -2.0 * a * b * safe ** (b - 1.0) / (1.0 + a * safe ** b), 0.0)


def _rep_coef_v(d2: np.ndarray, a: float, b: float) -> np.ndarray:
    """d/dy_i log(1 - Phi), regularised: c = 2b / ((1e-3 + d2)(1 + a d2^b)); 0 at d2 = 0."""
    safe = np.where(d2 > 0, d2, 1.0)
    return np.where(d2 > 0, 2.0 * b / ((1e-3 + safe) * (1.0 + a * safe ** b)), 0.0)


def frozen_epoch(g: Graph, E: np.ndarray, T: np.ndarray, epoch_idx: int, a: float, b: float, n_epochs: int,
                 neg_rate: int, seed: int, attr_mult: float = 1.0, self_skip: bool = False):
    """One epoch-synchronous step in which only the rows of g move (pull form,
    fp64): for every sampled edge e = (i, j), y_i gains alpha * attr_mult *
    clip(attraction toward T_j), and for each of its neg_rate draws k from
    [0, n_table) alpha * clip(repulsion from T_k).  A transform uses
    attr_mult = 1 and T the frozen layout; with T = E, attr_mult = 2 and draws
    equal to the source skipped this is the fit's epoch (each row also takes
    the equal share of its reverse edge).  Returns (E', sampled edges)."""
    E64 = np.asarray(E, dtype=np.float64)
    T64 = np.asarray(T, dtype=np.float64)
    alpha = 1.0 - epoch_idx / n_epochs
    e_act = np.nonzero(active_mask(g.eps, epoch_idx))[0]
    i = g.heads()[e_act].astype(np.int64)
    j = g.col[e_act].astype(np.int64)
    delta = np.zeros_like(E64)
    diff = E64[i] - T64[j]
    d2 = (diff * diff).sum(1)
    np.add.at(delta, i, alpha * attr_mult * np.clip(_attr_coef_v(d2, a, b)[:, None] * diff, -4.0, 4.0))
    if neg_rate > 0 and e_act.size:
        ks = negative_vertices(seed, epoch_idx, 0, g.nnz, neg_rate, T64.shape[0])[e_act].astype(np.int64)
        for r in range(neg_rate):
            k = ks[:, r]
            sel = k != i if self_skip else np.ones(k.size, dtype=bool)
            diff = E64[i[sel]] - T64[k[sel]]
            d2 = (diff * diff).sum(1)
            np.add.at(delta, i[sel], alpha * np.clip(_rep_coef_v(d2, a, b)[:, None] * diff, -4.0, 4.0))
    return E64 + delta, int(e_act.size)


def transform_run(g: Graph, T: np.ndarray, a: float, b: float, n_epochs: int, neg_rate: int, seed: int):
    """transform_init, then n_epochs frozen epochs.  Returns (Y_N, sampled edges per epoch)."""
    Y = transform_init(g, T)
    act = np.empty(n_epochs, dtype=np.int64)
    for ep in range(n_epochs):
        Y, act[ep] = frozen_epoch(g, Y, T, ep, a, b, n_epochs, neg_rate, seed)
    return Y, act


def exact_knn_cross(Q: np.ndarray, X: np.ndarray, k: int, batch: int = 1024) -> tuple[np.ndarray, np.ndarray]:
    """k nearest rows of X for every row of Q (Euclidean, fp64, ties by smaller
    index): the kNN query of new points against the kept training index."""
    Q64 = Q.astype(np.float64)
    X64 = X.astype(np.float64)
    ids = np.empty((Q.shape[0], k), dtype=np.int32)
    dist = np.empty((Q.shape[0], k), dtype=np.float32)
    for s in range(0, Q.shape[0], batch):
        t = min(Q.shape[0], s + batch)
        D = _sqdist(Q64[s:t], X64)
        cand = np.argpartition(D, k, axis=1)[:, : k + 1]
        diff = Q64[s:t, None, :] - X64[cand]
        ed = np.sqrt((diff * diff).sum(-1))
        order = np.lexsort((cand, ed), axis=1)[:, :k]
        ids[s:t] = np.take_along_axis(cand, order, axis=1)
        dist[s:t] = np.take_along_axis(ed, order, axis=1)
    return ids, dist
