"""Seeded synthetic inputs for the UMAP layout path.

This module only draws random numbers and lays them out; it performs none of
the method's arithmetic (no neighbour weighting, no union, no layout step), so
both the GPU path and the CPU oracle may take their inputs from it.

Workloads (the paper's datasets are not available, so seeded stand-ins of the
same shape are used; see the experiments section, dataset table):

* ``blobs2k``     2,000 points in 16-D, 5 isotropic Gaussian blobs (std 1,
                  centres uniform in [-10, 10]^16); stands in for the small
                  sets (digits, COIL-20) and the isotropic blobs of the
                  trustworthiness timing table.  Exact kNN, k = 15.
* ``image70k``    70,000 points in 784-D, 10 clusters; centre entries are 0
                  with probability 0.8, else U(0, 1); x = clip(N(c, 0.3), 0, 1).
                  Stands in for MNIST / Fashion-MNIST.  Exact kNN, k = 15.
* ``window1m``    1,000,000 vertices, a synthetic kNN graph: 30 contiguous
                  clusters of equal size; each vertex draws k = 15 distinct
                  neighbours uniformly from {i-64..i+64} inside its cluster,
                  with distances the running sum of k Exp(1) draws in draw
                  order.  Stands in for a pre-computed kNN graph at the
                  GoogleNews scale.
* ``window1m_k30`` as above with k = 30, 100 clusters and a 3-D embedding.
* ``window5m``    5,000,000 vertices, k = 15, 300 clusters with log-normal
                  (sigma 1) sizes rescaled to sum to n, each at least 129.
* ``window20m``, ``window50m``  the window1m recipe at 20M and 50M vertices
                  (600 and 1,500 equal clusters), for measurement at scale.
"""

from __future__ import annotations

import dataclasses

import numpy as np

WINDOW = 64          # neighbours are drawn from i-64 .. i+64 inside the cluster
_BLOCK = 1 << 16     # rows per generator block (fixed: part of the recipe)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n: int
    k: int
    dim: int
    n_epochs: int
    neg_rate: int
    min_dist: float
    spread: float
    seed: int           # numpy default_rng seed of the data generator
    kind: str           # "points" (exact kNN needed) or "window" (kNN drawn here)
    clusters: int = 0
    features: int = 0


WORKLOADS = {
    "blobs2k": Workload("blobs2k", 2000, 15, 2, 500, 5, 0.1, 1.0, 1, "points", 5, 16),
    "image70k": Workload("image70k", 70000, 15, 2, 200, 5, 0.1, 1.0, 2, "points", 10, 784),
    "window1m": Workload("window1m", 1_000_000, 15, 2, 200, 5, 0.1, 1.0, 3, "window", 30),
    "window1m_k30": Workload("window1m_k30", 1_000_000, 30, 3, 200, 5, 0.1, 1.0, 4, "window", 100),
    "window5m": Workload("window5m", 5_000_000, 15, 2, 200, 5, 0.1, 1.0, 5, "window", 300),
    # measurement only (no stored oracle runs): the 2-D table outgrows L2 (20M: 160 MB, inside the 256 MB
    # Infinity Cache) and then the Infinity Cache too (50M: 400 MB)
    "window20m": Workload("window20m", 20_000_000, 15, 2, 200, 5, 0.1, 1.0, 8, "window", 600),
    "window50m": Workload("window50m", 50_000_000, 15, 2, 200, 5, 0.1, 1.0, 9, "window", 1500),
}


def blobs(n: int = 2000, d: int = 16, centers: int = 5, seed: int = 1) -> tuple[np.ndarray, np.ndarray]:
    """Isotropic Gaussian blobs: equal-size groups around uniform centres."""
    rng = np.random.default_rng(seed)
    c = rng.uniform(-10.0, 10.0, size=(centers, d))
    labels = np.repeat(np.arange(centers), n // centers)
    labels = np.concatenate([labels, np.arange(n - labels.size) % centers])
    x = c[labels] + rng.standard_normal((n, d))
    return x.astype(np.float32), labels.astype(np.int32)


def image_like(n: int = 70000, d: int = 784, clusters: int = 10, seed: int = 2) -> tuple[np.ndarray, np.ndarray]:
    """Sparse non-negative image-like vectors clipped to [0, 1]."""
    rng = np.random.default_rng(seed)
    nz = rng.random((clusters, d)) >= 0.8
    c = np.where(nz, rng.random((clusters, d)), 0.0)
    labels = np.repeat(np.arange(clusters), n // clusters)
    labels = np.concatenate([labels, np.arange(n - labels.size) % clusters])
    x = np.empty((n, d), dtype=np.float32)
    for s in range(0, n, 8192):
        t = min(n, s + 8192)
        blk = c[labels[s:t]] + 0.3 * rng.standard_normal((t - s, d))
        x[s:t] = np.clip(blk, 0.0, 1.0)
    return x, labels.astype(np.int32)


def cluster_bounds(n: int, clusters: int, lognormal_sigma: float = 0.0, seed: int = 0,
                   min_size: int = 2 * WINDOW + 1) -> np.ndarray:
    """Start offsets (length clusters + 1) of contiguous clusters covering 0..n."""
    if lognormal_sigma <= 0.0:
        return (np.arange(clusters + 1, dtype=np.int64) * n) // clusters
    rng = np.random.default_rng(seed)
    w = np.exp(lognormal_sigma * rng.standard_normal(clusters))
    spare = n - min_size * clusters
    if spare < 0:
        raise ValueError("n too small for the requested clusters")
    sizes = min_size + np.floor(w / w.sum() * spare).astype(np.int64)
    sizes[: n - int(sizes.sum())] += 1          # distribute the rounding remainder
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


def window_knn(n: int, k: int, bounds: np.ndarray, seed: int, progress=None) -> tuple[np.ndarray, np.ndarray]:
    """Synthetic kNN lists: k distinct neighbours per vertex, drawn uniformly
    without replacement from the +-WINDOW window inside the vertex's cluster.
    Distances are the running sum of k Exp(1) draws, in draw order.
    `progress(rows_done)`, if given, is called after each block of rows.

    Returns ids (n, k) int32 and distances (n, k) float32.
    """
    rng = np.random.default_rng(seed)
    offs = np.concatenate([np.arange(-WINDOW, 0), np.arange(1, WINDOW + 1)])  # 128 candidates
    cl = np.searchsorted(bounds, np.arange(n), side="right") - 1
    ids = np.empty((n, k), dtype=np.int32)
    dist = np.empty((n, k), dtype=np.float32)
    for s in range(0, n, _BLOCK):
        t = min(n, s + _BLOCK)
        rows = np.arange(s, t)
        cand = rows[:, None] + offs[None, :]
        lo = bounds[cl[s:t]][:, None]
        hi = bounds[cl[s:t] + 1][:, None]
        ok = (cand >= lo) & (cand < hi)
        if np.any(ok.sum(axis=1) < k):
            raise ValueError("a cluster is too small for k distinct window neighbours")
        key = rng.random(cand.shape)
        key[~ok] = 2.0
        part = np.argpartition(key, k - 1, axis=1)[:, :k]
        order = np.argsort(np.take_along_axis(key, part, axis=1), axis=1, kind="stable")
        pick = np.take_along_axis(part, order, axis=1)              # draw order
        ids[s:t] = np.take_along_axis(cand, pick, axis=1)
        dist[s:t] = np.cumsum(rng.exponential(1.0, size=(t - s, k)), axis=1)
        if progress is not None:
            progress(t)
    return ids, dist


def workload_knn(w: Workload, progress=None) -> tuple[np.ndarray, np.ndarray]:
    """kNN ids/distances for a window workload."""
    if w.kind != "window":
        raise ValueError(f"{w.name} needs an exact kNN of its points")
    if w.name == "window5m":
        bounds = cluster_bounds(w.n, w.clusters, lognormal_sigma=1.0, seed=w.seed + 100)
    else:
        bounds = cluster_bounds(w.n, w.clusters)
    return window_knn(w.n, w.k, bounds, w.seed, progress)


def workload_points(w: Workload) -> tuple[np.ndarray, np.ndarray]:
    """Point cloud of a points workload."""
    if w.name == "blobs2k":
        return blobs(w.n, w.features, w.clusters, w.seed)
    if w.name == "image70k":
        return image_like(w.n, w.features, w.clusters, w.seed)
    raise ValueError(f"{w.name} has no point cloud")


def embedding_state(n: int, dim: int, seed: int, scale: float = 10.0) -> np.ndarray:
    """A seeded fp32 embedding state in [-scale, scale) (for single-epoch tests)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(-scale, scale, size=(n, dim)).astype(np.float32)


def random_symmetric_coo(n: int, avg_deg: int, seed: int, shuffle: bool = True):
    """A random symmetric weighted graph as COO (both directions listed, values
    bit-equal for (i, j) and (j, i)), in random order."""
    rng = np.random.default_rng(seed)
    m = max(1, n * avg_deg // 2)
    i = rng.integers(0, n, m)
    j = rng.integers(0, n, m)
    keep = i != j
    i, j = i[keep], j[keep]
    lo, hi = np.minimum(i, j), np.maximum(i, j)
    key = np.unique(lo.astype(np.int64) * n + hi)
    lo, hi = (key // n).astype(np.int32), (key % n).astype(np.int32)
    v = rng.random(lo.size).astype(np.float32) * np.float32(0.999) + np.float32(0.001)
    rows = np.concatenate([lo, hi])
    cols = np.concatenate([hi, lo])
    vals = np.concatenate([v, v])
    if shuffle:
        p = rng.permutation(rows.size)
        rows, cols, vals = rows[p], cols[p], vals[p]
    return rows, cols, vals


def quality_sample(n: int, rows: int = 10_000, negatives: int = 64, seed: int = 12345):
    """Seeded vertex sample for the quality measures of graph-only workloads:
    `rows` distinct vertices (sorted) and, for each, `negatives` vertices drawn
    uniformly from [0, n) (the fixed stand-ins of the objective's random
    negative samples)."""
    rng = np.random.default_rng(seed)
    r = np.sort(rng.choice(n, size=min(rows, n), replace=False)).astype(np.int64)
    neg = rng.integers(0, n, size=(r.size, negatives), dtype=np.int64)
    return r, neg


def transform_graph(n_new: int, n_table: int, k: int = 15, seed: int = 6):
    """Bipartite COO graph of n_new new points against n_table laid-out
    vertices, for timing a transform: each new point picks an anchor row a
    uniformly in [64, n_table - 65) and k distinct neighbours uniformly from
    a - 64 .. a + 64, with weights uniform on [0.05, 1)."""
    if n_table < 2 * WINDOW + 2:
        raise ValueError("the table needs at least 130 rows")
    rng = np.random.default_rng(seed)
    anchor = rng.integers(WINDOW, n_table - WINDOW - 1, size=(n_new, 1))
    rows = np.repeat(np.arange(n_new, dtype=np.int32), k)
    cols = np.empty((n_new, k), dtype=np.int32)
    for s in range(0, n_new, _BLOCK):
        t = min(n_new, s + _BLOCK)
        off = np.argsort(rng.random((t - s, 2 * WINDOW + 1)), axis=1)[:, :k] - WINDOW
        cols[s:t] = (anchor[s:t] + off).astype(np.int32)
    vals = rng.uniform(0.05, 1.0, size=rows.size).astype(np.float32)
    return rows, cols.ravel(), vals
