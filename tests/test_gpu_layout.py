"""GPU parity of the layout path against the CPU oracle (MI355X, gfx950).

Every test goes through the C ABI (ctypes binding) and compares with the
oracle on the same seeded inputs:
  * the ingested graph (row_ptr, col, eps): bit-exact;
  * the schedule (active edges per epoch) and the negative-sample draws:
    bit-exact;
  * the random initial layout: bit-exact;
  * one epoch fed the same fp32 state: max |GPU - oracle| <= 1e-4;
  * a full run: trustworthiness at k = 15 within 0.01 of the oracle's run;
  * determinism, resume and the two epoch kernels: bit-identical.
"""

import sys

import time

import numpy as np
import pytest

import oracle as O
from paper_2008_00325_amd import synth
from paper_2008_00325_amd import umap_layout as U

pytestmark = pytest.mark.gpu

TOL = 1e-4
A_DEF, B_DEF = 1.5769434, 0.8950608


@pytest.fixture(scope="module", autouse=True)
def torch_device_first():
    """Initialise torch's HIP runtime before the library's (torch ships its own
    copy of the runtime; the tests use torch tensors for device memory)."""
    import torch

    torch.cuda.init()
    torch.cuda.set_device(0)


def case(msg):
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def _coo_from_knn(ids, dist):
    return O.fuzzy_graph(ids, dist)


@pytest.fixture(scope="module")
def blobs_graph():
    w = synth.WORKLOADS["blobs2k"]
    X, _ = synth.workload_points(w)
    ids, dist = O.exact_knn(X, w.k)
    r, c, v = _coo_from_knn(ids, dist)
    return w, X, ids, dist, (r, c, v)


@pytest.fixture(scope="module")
def window1m_graph():
    w = synth.WORKLOADS["window1m"]
    ids, dist = synth.workload_knn(w)
    r, c, v = _coo_from_knn(ids, dist)
    return w, ids, dist, (r, c, v)


def _shuffled(coo, seed):
    r, c, v = coo
    p = np.random.default_rng(seed).permutation(r.size)
    return r[p], c[p], v[p]


def _check_graph(h, g):
    row_ptr, col, eps = U.umap_layout_get_graph(h)
    assert np.array_equal(row_ptr, g.row_ptr)
    assert np.array_equal(col, g.col)
    assert np.array_equal(eps.view(np.uint32), g.eps.view(np.uint32))
    st = U.umap_layout_stats(h)
    assert st["nnz_kept"] == g.nnz and np.float32(st["w_max"]) == np.float32(g.w_max)


# ---------------------------------------------------------------------------
# ingest
# ---------------------------------------------------------------------------

def test_graph_bit_exact_host_and_device(blobs_graph):
    import torch

    w, X, ids, dist, coo = blobs_graph
    r, c, v = _shuffled(coo, 1)
    # zeros, negatives and self loops must be dropped
    r = np.concatenate([r, [3, 4, 5]]).astype(np.int32)
    c = np.concatenate([c, [3, 9, 6]]).astype(np.int32)
    v = np.concatenate([v, [0.7, 0.0, -1.0]]).astype(np.float32)
    g = O.prep(w.n, r, c, v, w.n_epochs)
    case("graph blobs2k host create")
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, w.n_epochs, 5) as h:
        _check_graph(h, g)
    case("graph blobs2k device create")
    dr, dc, dv = (torch.from_numpy(x).cuda() for x in (r, c, v))
    with U.umap_layout_create_device(w.n, 2, dr, dc, dv, r.size, A_DEF, B_DEF, w.n_epochs, 5) as h:
        _check_graph(h, g)


@pytest.mark.parametrize("n,deg,N", [(1, 0, 10), (7, 3, 1), (3001, 9, 200), (20011, 30, 50)])
def test_graph_bit_exact_random(n, deg, N):
    if deg == 0:
        r = c = np.zeros(0, np.int32)
        v = np.zeros(0, np.float32)
    else:
        r, c, v = synth.random_symmetric_coo(n, deg, seed=n)
    g = O.prep(n, r, c, v, N)
    case(f"graph random n={n} deg={deg} N={N}")
    with U.umap_layout_create(n, 3, r, c, v, A_DEF, B_DEF, N, 5) as h:
        _check_graph(h, g)


@pytest.mark.parametrize("n", [6000, 40001])
def test_graph_hub_row(n):
    """A star: vertex 0 joined to every other vertex (a row of n - 1 edges; at
    40,001 vertices longer than a wave's whole cost, so the row is a wave of its
    own), both kernels; the asynchronous mode's sampled-edge count and a finite
    result."""
    others = np.arange(1, n, dtype=np.int32)
    vals = np.random.default_rng(3).random(n - 1).astype(np.float32) + np.float32(0.01)
    r = np.concatenate([np.zeros(n - 1, np.int32), others])
    c = np.concatenate([others, np.zeros(n - 1, np.int32)])
    v = np.concatenate([vals, vals])
    r, c, v = _shuffled((r, c, v), 2)
    g = O.prep(n, r, c, v, 100)
    case(f"graph star n={n}")
    with U.umap_layout_create(n, 2, r, c, v, A_DEF, B_DEF, 100, 5) as h:
        _check_graph(h, g)
        assert U.umap_layout_stats(h)["max_degree"] == int(np.diff(g.row_ptr).max()) > 8192 * (n > 10000)
        E = synth.embedding_state(n, 2, 9)
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for ep in (0, 50, 99):
                case(f"graph star n={n} kernel {kernel} epoch {ep}")
                U.umap_layout_set_embedding(h, E)
                U.umap_layout_run_epochs(h, 4, ep, ep + 1)
                ref, act = O.epoch(g, E, ep, A_DEF, B_DEF, 100, 5, 4)
                assert np.abs(U.umap_layout_get(h) - ref).max() <= TOL
                st = U.umap_layout_stats(h)
                assert st["active_edges"] == act and st["overflow_redone"] == 0
        U.umap_layout_set_mode(h, U.UMAP_MODE_ASYNC)
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, 4, 0, 10)
            assert np.all(np.isfinite(U.umap_layout_get(h)))
            assert U.umap_layout_stats(h)["active_edges"] == sum(
                int(O.active_mask(g.eps, ep).sum()) for ep in range(10))


def _stars(n, hubs, seed):
    """Symmetric COO: each hub h joined to `size` distinct random other
    vertices (bit-equal values both ways), plus a sparse random graph."""
    rng = np.random.default_rng(seed)
    pairs = {}
    for h, size in hubs:
        others = rng.choice(np.delete(np.arange(n), h), size=size, replace=False)
        for j in others:
            pairs[(min(h, int(j)), max(h, int(j)))] = None
    r0, c0, _ = synth.random_symmetric_coo(n, 4, seed=seed + 1, shuffle=False)
    for a, b in zip(r0, c0):
        if a < b:
            pairs[(int(a), int(b))] = None
    lo = np.array([p[0] for p in pairs], np.int32)
    hi = np.array([p[1] for p in pairs], np.int32)
    v = (rng.random(lo.size).astype(np.float32) + np.float32(0.01))
    return np.concatenate([lo, hi]), np.concatenate([hi, lo]), np.concatenate([v, v])


def test_graph_long_rows():
    """Rows longer than the rank sort's limit go through the per-row radix
    sort: a star whose hub has 2^20 edges ingests bit-exact against the
    oracle in bounded time (the rank sort would read the hub row 2^40 times),
    host and device create; hubs of 2,049 to 70,000 edges among ordinary rows;
    a duplicate inside a long row is reported."""
    import torch

    n = (1 << 20) + 1
    others = np.arange(1, n, dtype=np.int32)
    vals = np.random.default_rng(5).random(n - 1).astype(np.float32) + np.float32(0.01)
    r = np.concatenate([np.zeros(n - 1, np.int32), others])
    c = np.concatenate([others, np.zeros(n - 1, np.int32)])
    v = np.concatenate([vals, vals])
    r, c, v = _shuffled((r, c, v), 6)
    g = O.prep(n, r, c, v, 200)
    case("graph star with a 2^20-edge hub, host create")
    with U.umap_layout_create(n, 2, r, c, v, A_DEF, B_DEF, 200, 5) as h:
        _check_graph(h, g)
        st = U.umap_layout_stats(h)
        print(f"  ingest {st['prep_ms']:.2f} ms, max degree {st['max_degree']}", flush=True)
        assert st["max_degree"] == n - 1 and st["prep_ms"] < 500.0
    case("graph star with a 2^20-edge hub, device create")
    dr, dc, dv = (torch.from_numpy(x).cuda() for x in (r, c, v))
    with U.umap_layout_create_device(n, 2, dr, dc, dv, r.size, A_DEF, B_DEF, 200, 5) as h:
        _check_graph(h, g)
    n2 = 200_003
    r, c, v = _stars(n2, [(7, 2075), (100_000, 3000), (199_999, 10_000), (5, 70_000), (6, 2048)], 9)
    r, c, v = _shuffled((r, c, v), 10)
    g = O.prep(n2, r, c, v, 50)
    assert np.diff(g.row_ptr)[7] > 2048 >= np.diff(g.row_ptr)[6]
    case("graph with hubs of 2,048 to 70,000 edges")
    with U.umap_layout_create(n2, 3, r, c, v, A_DEF, B_DEF, 50, 5) as h:
        _check_graph(h, g)
    case("duplicate inside a long row")
    # one extra (5, j): only the long row 5 holds a duplicate
    dup = np.flatnonzero((r == 5) & (c != 6))[:1]
    r2 = np.concatenate([r, r[dup]])
    c2 = np.concatenate([c, c[dup]])
    v2 = np.concatenate([v, v[dup]])
    with pytest.raises(U.UmapLayoutError) as ei:
        U.umap_layout_create(n2, 3, r2, c2, v2, A_DEF, B_DEF, 50, 5)
    assert ei.value.code == U.UMAP_E_INVAL and "more than once" in U.umap_layout_last_error()


def test_graph_errors_on_device():
    import torch

    r = np.array([0, 1, 1, 2], np.int32)
    c = np.array([1, 0, 2, 1], np.int32)
    case("asymmetric value")
    with pytest.raises(U.UmapLayoutError) as ei:
        U.umap_layout_create(3, 2, r, c, np.float32([0.5, 0.5, 0.5, 0.25]), A_DEF, B_DEF, 10, 5)
    assert ei.value.code == U.UMAP_E_ASYMMETRIC
    case("missing reverse edge")
    with pytest.raises(U.UmapLayoutError) as ei:
        U.umap_layout_create(3, 2, r[:3], c[:3], np.float32([0.5, 0.5, 0.5]), A_DEF, B_DEF, 10, 5)
    assert ei.value.code == U.UMAP_E_ASYMMETRIC
    case("duplicate edge")
    with pytest.raises(U.UmapLayoutError) as ei:
        U.umap_layout_create(3, 2, np.r_[r, 0], np.r_[c, 1], np.float32([0.5] * 5), A_DEF, B_DEF, 10, 5)
    assert ei.value.code == U.UMAP_E_INVAL and "more than once" in U.umap_layout_last_error()
    case("device path: index out of range and non-finite value")
    for rr, vv, frag in [(np.int32([0, 1, 1, 7]), np.float32([0.5] * 4), "outside"),
                         (r, np.float32([0.5, np.nan, 0.5, 0.5]), "not finite")]:
        dr, dc, dv = (torch.from_numpy(x).cuda() for x in (rr, c, vv))
        with pytest.raises(U.UmapLayoutError) as ei:
            U.umap_layout_create_device(3, 2, dr, dc, dv, 4, A_DEF, B_DEF, 10, 5)
        assert ei.value.code == U.UMAP_E_INVAL and frag in U.umap_layout_last_error()


# ---------------------------------------------------------------------------
# schedule, random streams, initial layout
# ---------------------------------------------------------------------------

def test_active_mask_and_negatives_bit_exact(blobs_graph):
    w, X, ids, dist, (r, c, v) = blobs_graph
    g = O.prep(w.n, r, c, v, w.n_epochs)
    case("active mask / negatives blobs2k")
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, w.n_epochs, 5) as h:
        for ep in (0, 1, 2, 3, w.n_epochs // 2, w.n_epochs - 1):
            assert np.array_equal(U.umap_layout_debug_active(h, ep), O.active_mask(g.eps, ep))
        for seed, ep, e0 in [(0, 0, 0), (2**40 + 7, 17, 1234), (2**64 - 1, w.n_epochs - 1, g.nnz - 500)]:
            got = U.umap_layout_debug_negatives(h, seed, ep, e0, 500)
            ref = O.negative_vertices(seed, ep, e0, 500, 5, w.n)
            assert np.array_equal(got, ref)


@pytest.mark.parametrize("n,dim", [(1, 1), (1000, 2), (4097, 3), (3000, 16)])
def test_init_bit_exact(n, dim):
    case(f"init n={n} dim={dim}")
    empty = np.zeros(0, np.int32)
    with U.umap_layout_create(n, dim, empty, empty, np.zeros(0, np.float32), A_DEF, B_DEF, 3, 5) as h:
        for seed in (0, 12345, 2**63 + 5):
            U.umap_layout_run(h, seed)
            assert np.array_equal(U.umap_layout_get(h).view(np.uint32), O.init_layout(n, dim, seed).view(np.uint32))
            assert U.umap_layout_stats(h)["active_edges"] == 0


# ---------------------------------------------------------------------------
# one epoch from the same state
# ---------------------------------------------------------------------------

def _epoch_parity(h, g, E, epochs, a, b, N, R, seed, label):
    for ep in epochs:
        case(f"{label} epoch {ep}")
        U.umap_layout_set_embedding(h, E)
        U.umap_layout_run_epochs(h, seed, ep, ep + 1)
        got = U.umap_layout_get(h)
        ref, act = O.epoch(g, E, ep, a, b, N, R, seed)
        err = float(np.abs(got.astype(np.float64) - ref).max())
        print(f"  max|diff| = {err:.3e}  active = {act}", flush=True)
        assert err <= TOL
        st = U.umap_layout_stats(h)
        assert st["active_edges"] == act
        assert st["overflow_redone"] == 0


def test_single_epoch_blobs(blobs_graph):
    w, X, ids, dist, (r, c, v) = blobs_graph
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    # the oracle's own trajectory, rounded to fp32, as the fed states
    E0 = O.init_layout(w.n, 2, 7).astype(np.float64)
    states = [E0]
    E = E0
    for ep in range(30):
        E, _ = O.epoch(g, E, ep, a, b, w.n_epochs, w.neg_rate, 7)
    states.append(E)
    with U.umap_layout_create(w.n, 2, r, c, v, a, b, w.n_epochs, w.neg_rate) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for s in states:
                _epoch_parity(h, g, s.astype(np.float32), (0, 1, w.n_epochs // 2, w.n_epochs - 1), a, b,
                              w.n_epochs, w.neg_rate, 7, f"blobs2k kernel {kernel}")


def test_single_epoch_window1m_full_size(window1m_graph):
    """The workload the benchmark times (1M vertices, k = 15, 2-D), whole
    layout compared, in the benchmark's launch configuration."""
    import torch

    w, ids, dist, (r, c, v) = window1m_graph
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    dr, dc, dv = (torch.from_numpy(x).cuda() for x in (r, c, v))
    with U.umap_layout_create_device(w.n, w.dim, dr, dc, dv, r.size, a, b, w.n_epochs, w.neg_rate) as h:
        _check_graph(h, g)
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for scale, seed in ((10.0, 3), (0.5, 4)):
                E = synth.embedding_state(w.n, w.dim, seed, scale)
                _epoch_parity(h, g, E, (0, 1, w.n_epochs // 2, w.n_epochs - 1), a, b, w.n_epochs, w.neg_rate, 11,
                              f"window1m kernel {kernel} scale {scale}")


@pytest.mark.parametrize("name", ["window1m_k30", "window5m"])
def test_single_epoch_other_full_sizes(name):
    """The two other full-size workloads: 1M vertices with k = 30 in 3-D (4
    table ranges) and 5M vertices with lognormal cluster sizes (8 table
    ranges); whole layout compared after one epoch fed the same fp32 state."""
    import torch

    w = synth.WORKLOADS[name]
    case(f"{name}: building the graph on the host")
    ids, dist = synth.workload_knn(w)
    r, c, v = O.fuzzy_graph(ids, dist)
    del ids, dist
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    dr, dc, dv = (torch.from_numpy(x).cuda() for x in (r, c, v))
    nnz = r.size
    del r, c, v
    with U.umap_layout_create_device(w.n, w.dim, dr, dc, dv, nnz, a, b, w.n_epochs, w.neg_rate) as h:
        del dr, dc, dv
        _check_graph(h, g)
        st = U.umap_layout_stats(h)
        case(f"{name}: {st['table_ranges']} table ranges, {st['nnz_kept']} edges")
        assert st["table_ranges"] == (4 if w.n == 1_000_000 else 8)
        E = synth.embedding_state(w.n, w.dim, 6, 10.0)
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            _epoch_parity(h, g, E, (0, 1, w.n_epochs // 2, w.n_epochs - 1), a, b, w.n_epochs, w.neg_rate, 13,
                          f"{name} kernel {kernel} scale 10")


def test_sixteen_table_ranges_sampled_rows():
    """Past 5M vertices the table is split into 16 ranges: a sparse random
    graph of 5.2M vertices, one epoch from a seeded state, 20,000 sampled
    rows against the oracle's update of those rows (both kernels)."""
    n, N, R, seed = 5_200_000, 50, 5, 17
    case(f"{n} vertices: building a random graph")
    r, c, v = synth.random_symmetric_coo(n, 4, 31)
    g = O.prep(n, r, c, v, N)
    E = synth.embedding_state(n, 2, 9, 10.0)
    rows = np.sort(np.random.default_rng(5).choice(n, size=20_000, replace=False)).astype(np.int64)
    with U.umap_layout_create(n, 2, r, c, v, A_DEF, B_DEF, N, R) as h:
        assert U.umap_layout_stats(h)["table_ranges"] == 16
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for ep in (0, N // 2):
                case(f"{n} vertices, 16 ranges, kernel {kernel} epoch {ep}")
                U.umap_layout_set_embedding(h, E)
                U.umap_layout_run_epochs(h, seed, ep, ep + 1)
                got = U.umap_layout_get(h)
                st = U.umap_layout_stats(h)
                assert st["overflow_redone"] == 0
                assert st["active_edges"] == int(O.active_mask(g.eps, ep).sum())
                ref = E[rows].astype(np.float64) + O.epoch_rows(g, E, ep, A_DEF, B_DEF, N, R, seed, rows)
                err = float(np.abs(got[rows].astype(np.float64) - ref).max())
                print(f"  max|diff| = {err:.3e}", flush=True)
                assert err <= TOL


def _window_quality_golden():
    import json
    import os

    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "window_quality.json")
    with open(path) as f:
        return json.load(f)


@pytest.mark.parametrize("name,mode,kernel", [("window1m", 0, 0), ("window1m", 1, 0), ("window1m", 1, 1),
                                               ("window1m_k30", 0, 0), ("window5m", 0, 0)])
def test_full_run_quality_window(name, mode, kernel):
    """Full 200-epoch runs of the graph-only workloads, scored like the oracle's
    stored runs (same seed, same sample): recall@15 within 0.01 and the
    objective within 1 % of the oracle's.  The asynchronous mode (a different
    trajectory, not the oracle's) must be no worse by the same margins."""
    import torch

    gold = _window_quality_golden()
    if name not in gold:
        pytest.skip(f"no stored oracle run for {name} (tests/golden/make_window_quality.py writes it)")
    ref = gold[name]
    seed = gold["seed"]
    w = synth.WORKLOADS[name]
    case(f"{name} mode {mode}: building the graph on the host")
    ids, dist = synth.workload_knn(w)
    r, c, v = O.fuzzy_graph(ids, dist)
    del dist
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    dr, dc, dv = (torch.from_numpy(x).cuda() for x in (r, c, v))
    nnz = r.size
    del r, c, v
    case(f"{name} mode {mode} kernel {kernel}: GPU run")
    with U.umap_layout_create_device(w.n, w.dim, dr, dc, dv, nnz, a, b, w.n_epochs, w.neg_rate) as h:
        del dr, dc, dv
        U.umap_layout_set_mode(h, mode)
        U.umap_layout_set_kernel(h, kernel)
        U.umap_layout_run(h, seed)
        E = U.umap_layout_get(h)
        st = U.umap_layout_stats(h)
    assert st["active_edges"] == ref["active_edges"]
    assert np.all(np.isfinite(E))
    rows, neg = synth.quality_sample(w.n)
    rec = O.recall_at_k(ids, E, rows, 15)
    obj = O.objective(g, E, a, b, w.neg_rate, rows, neg)
    print(f"  recall@15 {rec:.4f} (oracle {ref['recall15']:.4f}, init {ref['recall15_init']:.4f}); "
          f"objective {obj:.6g} (oracle {ref['objective']:.6g}, init {ref['objective_init']:.6g})", flush=True)
    if mode == U.UMAP_MODE_SYNC:
        assert abs(rec - ref["recall15"]) <= 0.01
        assert abs(obj - ref["objective"]) <= 0.01 * ref["objective"]
    else:
        # in-place updates let later edges of an epoch see earlier moves: the
        # asynchronous run may converge further than the oracle's synchronous
        # one, so its bound is one-sided (no worse than the oracle's)
        assert rec >= ref["recall15"] - 0.01
        assert obj <= 1.01 * ref["objective"]


@pytest.mark.parametrize("dim,R,N", [(1, 5, 20), (3, 5, 200), (4, 0, 50), (6, 5, 25), (16, 7, 30), (2, 12, 40)])
def test_single_epoch_dims_and_rates(dim, R, N):
    n = 5003
    bounds = synth.cluster_bounds(n, 3)
    ids, dist = synth.window_knn(n, 15, bounds, seed=dim)
    r, c, v = O.fuzzy_graph(ids, dist)
    g = O.prep(n, r, c, v, N)
    with U.umap_layout_create(n, dim, r, c, v, A_DEF, B_DEF, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for scale in (10.0, 0.3):
                E = synth.embedding_state(n, dim, dim + 100, scale)
                _epoch_parity(h, g, E, (0, 1, N // 2, N - 1), A_DEF, B_DEF, N, R, 5,
                              f"dim {dim} R {R} kernel {kernel} scale {scale}")


@pytest.mark.parametrize("dim", list(range(1, 17)))
def test_every_width_both_kernels(dim):
    # every embedding width on a locally ordered graph (all tails within +-64
    # rows): the wave kernels stage halo rows at 1-2 components and read other
    # tails from global memory, and pad the LDS rows of even widths from 4 on;
    # one epoch of each kernel must match the oracle and each other bit for bit
    n, N, R = 4001, 60, 5
    print(f"[gpu case] width {dim}", flush=True)
    ids, dist = synth.window_knn(n, 15, synth.cluster_bounds(n, 2), seed=40 + dim)
    r, c, v = O.fuzzy_graph(ids, dist)
    g = O.prep(n, r, c, v, N)
    E = synth.embedding_state(n, dim, 300 + dim, 10.0)
    ref, act = O.epoch(g, E, 7, A_DEF, B_DEF, N, R, 11)
    outs = []
    with U.umap_layout_create(n, dim, r, c, v, A_DEF, B_DEF, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, 11, 7, 8)
            got = U.umap_layout_get(h)
            assert float(np.abs(got.astype(np.float64) - ref).max()) <= TOL, (dim, kernel)
            assert U.umap_layout_stats(h)["active_edges"] == act
            outs.append(got)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32)), dim


@pytest.fixture(scope="module")
def window1m_prep(window1m_graph):
    w, ids, dist, (r, c, v) = window1m_graph
    return O.prep(w.n, r, c, v, w.n_epochs)


@pytest.mark.parametrize("dim", list(range(2, 17)))
def test_every_width_several_ranges(dim, window1m_graph, window1m_prep):
    # every width from 2 on with a table of several ranges (the 1M window
    # graph: 8 MB and more, 4 ranges), where the draw kernel files records and
    # the range launches apply them: 20,000 sampled rows of one epoch against
    # the oracle, and the two kernels bit for bit on the whole layout
    w, ids, dist, (r, c, v) = window1m_graph
    g = window1m_prep
    N, R, ep, seed = w.n_epochs, w.neg_rate, 9, 23
    print(f"[gpu case] width {dim}, 1M vertices, several table ranges", flush=True)
    E = synth.embedding_state(w.n, dim, 500 + dim, 10.0)
    rows = np.sort(np.random.default_rng(dim).choice(w.n, size=20_000, replace=False)).astype(np.int64)
    ref = E[rows].astype(np.float64) + O.epoch_rows(g, E, ep, A_DEF, B_DEF, N, R, seed, rows)
    outs = []
    with U.umap_layout_create(w.n, dim, r, c, v, A_DEF, B_DEF, N, R) as h:
        assert U.umap_layout_stats(h)["table_ranges"] == 4
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, seed, ep, ep + 1)
            got = U.umap_layout_get(h)
            st = U.umap_layout_stats(h)
            assert st["overflow_redone"] == 0
            assert st["active_edges"] == int(O.active_mask(g.eps, ep).sum())
            err = float(np.abs(got[rows].astype(np.float64) - ref).max())
            print(f"  kernel {kernel}: max|diff| = {err:.3e}", flush=True)
            assert err <= TOL, (dim, kernel)
            outs.append(got)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32)), dim


# ---------------------------------------------------------------------------
# whole runs
# ---------------------------------------------------------------------------

def test_kernels_bit_identical_and_deterministic(window1m_graph):
    w, ids, dist, (r, c, v) = window1m_graph
    sub = (r < 200_000) & (c < 200_000)
    r, c, v = r[sub], c[sub], v[sub]
    n = 200_000
    N = 20
    case("two kernels and two runs, 200k vertices, 20 epochs")
    with U.umap_layout_create(n, 2, r, c, v, A_DEF, B_DEF, N, 5) as h:
        U.umap_layout_run(h, 77)
        first = U.umap_layout_get(h)
        U.umap_layout_run(h, 77)
        assert np.array_equal(U.umap_layout_get(h).view(np.uint32), first.view(np.uint32))
        U.umap_layout_set_kernel(h, 1)
        U.umap_layout_run(h, 77)
        assert np.array_equal(U.umap_layout_get(h).view(np.uint32), first.view(np.uint32))
        U.umap_layout_set_kernel(h, 0)
        U.umap_layout_run(h, 78)
        assert not np.array_equal(U.umap_layout_get(h), first)


def test_epoch_timing(blobs_graph):
    """Per-epoch HIP events: off by default; on, one device time per epoch of
    the call whose sum is the call's epochs time, for any kernel; at most 4096
    epochs of a call are timed; bad arguments are rejected."""
    w, X, ids, dist, (r, c, v) = blobs_graph
    case("per-epoch timing, blobs2k")
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, 5000, w.neg_rate) as h:
        U.umap_layout_init(h, 3)
        U.umap_layout_run_epochs(h, 3, 0, 10)
        assert U.umap_layout_epoch_ms(h).size == 0
        U.umap_layout_set_epoch_timing(h, True)
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_run_epochs(h, 3, 20, 70)
            t = U.umap_layout_epoch_ms(h)
            st = U.umap_layout_stats(h)
            print(f"  kernel {kernel}: 50 epochs {t.sum():.3f} ms (call {st['epochs_ms']:.3f} ms), "
                  f"min {t.min():.4f} max {t.max():.4f}", flush=True)
            assert t.size == 50 and np.all(t > 0)
            assert t.sum() <= st["epochs_ms"] * 1.001 + 1e-3
            assert t.sum() >= 0.5 * st["epochs_ms"]
        U.umap_layout_run_epochs(h, 3, 0, 5000)
        assert U.umap_layout_epoch_ms(h).size == 4096
        buf = np.zeros(3, np.float32)
        assert U.lib().umap_layout_epoch_ms(h.ptr, buf.ctypes.data, 3) == 4096
        assert np.all(buf > 0)
        assert U.lib().umap_layout_epoch_ms(h.ptr, None, -1) == U.UMAP_E_INVAL
        assert U.lib().umap_layout_epoch_ms(h.ptr, None, 2) == U.UMAP_E_INVAL
        U.umap_layout_set_epoch_timing(h, False)
        U.umap_layout_run_epochs(h, 3, 0, 10)
        assert U.umap_layout_epoch_ms(h).size == 0


def test_two_handles_on_two_streams_in_parallel(window1m_graph):
    """Two host threads, each driving its own handle on its own stream at the
    same time (one with each kernel): every result equals the same run made
    alone, bit for bit -- the library keeps no shared mutable state."""
    import threading

    import torch

    w, ids, dist, (r, c, v) = window1m_graph
    sub = (r < 200_000) & (c < 200_000)
    r, c, v = r[sub], c[sub], v[sub]
    n, N = 200_000, 30
    seeds = (11, 12)
    alone = {}
    for s in seeds:
        case(f"two streams: seed {s} alone")
        with U.umap_layout_create(n, 2, r, c, v, A_DEF, B_DEF, N, 5) as h:
            U.umap_layout_run(h, s)
            alone[s] = U.umap_layout_get(h)
    got, errors = {}, []

    def worker(s, kernel):
        try:
            stream = torch.cuda.Stream()
            with U.umap_layout_create(n, 2, r, c, v, A_DEF, B_DEF, N, 5) as h:
                U.umap_layout_set_stream(h, stream)
                U.umap_layout_set_kernel(h, kernel)
                for _ in range(3):
                    U.umap_layout_run(h, s)
                got[s] = U.umap_layout_get(h)
        except Exception as e:  # reported by the main thread
            errors.append(e)

    case("two streams: both seeds in parallel")
    threads = [threading.Thread(target=worker, args=(s, k)) for s, k in zip(seeds, (0, 1))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
    for s in seeds:
        assert np.array_equal(got[s].view(np.uint32), alone[s].view(np.uint32))


def test_resume_equals_uninterrupted(blobs_graph):
    w, X, ids, dist, (r, c, v) = blobs_graph
    N = 60
    case("resume at epoch 23 of 60")
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, N, 5) as h:
        U.umap_layout_run(h, 5)
        full = U.umap_layout_get(h)
        U.umap_layout_set_embedding(h, O.init_layout(w.n, 2, 5))
        U.umap_layout_run_epochs(h, 5, 0, 23)
        mid = U.umap_layout_get(h)
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, N, 5) as h2:
        U.umap_layout_set_embedding(h2, mid)
        U.umap_layout_run_epochs(h2, 5, 23, N)
        assert np.array_equal(U.umap_layout_get(h2).view(np.uint32), full.view(np.uint32))
        # init, then the epochs in two pieces, equals one run
        U.umap_layout_init(h2, 5)
        assert np.array_equal(U.umap_layout_get(h2), O.init_layout(w.n, 2, 5))
        U.umap_layout_run_epochs(h2, 5, 0, 40)
        U.umap_layout_run_epochs(h2, 5, 40, N)
        assert np.array_equal(U.umap_layout_get(h2).view(np.uint32), full.view(np.uint32))


def test_full_run_trustworthiness(blobs_graph):
    w, X, ids, dist, (r, c, v) = blobs_graph
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    for seed in (0, 1):
        case(f"full run blobs2k seed {seed}")
        with U.umap_layout_create(w.n, w.dim, r, c, v, a, b, w.n_epochs, w.neg_rate) as h:
            U.umap_layout_run(h, seed)
            Eg = U.umap_layout_get(h)
            st = U.umap_layout_stats(h)
        t0 = time.perf_counter()
        Eo, act = O.run(g, w.dim, a, b, w.n_epochs, w.neg_rate, seed)
        to_s = time.perf_counter() - t0
        assert st["active_edges"] == int(act.sum())
        assert st["edge_updates"] == int(act.sum()) * (1 + w.neg_rate)
        tg = O.trustworthiness(X, Eg, 15)
        to = O.trustworthiness(X, Eo, 15)
        print(f"  T(gpu) = {tg:.5f}  T(oracle) = {to:.5f}; GPU epochs {st['epochs_ms']:.2f} ms "
              f"({st['edge_updates'] / (st['epochs_ms'] * 1e-3):.3e} edge-updates/s), oracle run {to_s:.2f} s "
              f"on {O.num_threads()} threads", flush=True)
        assert abs(tg - to) <= 0.01
        assert np.all(np.isfinite(Eg))


@pytest.mark.parametrize("kernel", [0, 1])
@pytest.mark.parametrize("dim,R", [(2, 5), (3, 5), (16, 10), (2, 0)])
def test_async_mode_quality(dim, R, kernel, blobs_graph):
    """Asynchronous (Hogwild) mode, the paper's default, with either kernel
    (0 range-ordered, 1 per-edge): not repeatable bit for bit, so the check is
    on quality -- T@15 of a full run within 0.01 of the oracle's
    (epoch-synchronous) run at the same settings -- plus the parts that stay
    deterministic (the number of sampled edges, the mode switch)."""
    w, X, ids, dist, (r, c, v) = blobs_graph
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    seed = 4
    case(f"async blobs2k dim {dim} R {R} kernel {kernel}")
    with U.umap_layout_create(w.n, dim, r, c, v, a, b, w.n_epochs, R) as h:
        U.umap_layout_run(h, seed)
        Es = U.umap_layout_get(h)
        U.umap_layout_set_mode(h, U.UMAP_MODE_ASYNC)
        U.umap_layout_set_kernel(h, kernel)
        U.umap_layout_run(h, seed)
        Ea = U.umap_layout_get(h)
        st = U.umap_layout_stats(h)
        assert st["mode"] == U.UMAP_MODE_ASYNC and st["overflow_redone"] == 0
        U.umap_layout_set_kernel(h, 0)
        with pytest.raises(U.UmapLayoutError) as ei:
            U.umap_layout_set_mode(h, 2)
        assert ei.value.code == U.UMAP_E_INVAL
        U.umap_layout_set_mode(h, U.UMAP_MODE_SYNC)
        U.umap_layout_run(h, seed)
        assert np.array_equal(U.umap_layout_get(h).view(np.uint32), Es.view(np.uint32))
    Eo, act = O.run(g, dim, a, b, w.n_epochs, R, seed)
    assert st["active_edges"] == int(act.sum())
    assert st["edge_updates"] == int(act.sum()) * (1 + R)
    assert np.all(np.isfinite(Ea))
    ta = O.trustworthiness(X, Ea, 15)
    to = O.trustworthiness(X, Eo, 15)
    print(f"  T(async) = {ta:.5f}  T(oracle) = {to:.5f}", flush=True)
    assert abs(ta - to) <= 0.01


def test_fault_injection(monkeypatch, blobs_graph):
    w, X, ids, dist, (r, c, v) = blobs_graph
    case("fault injection")
    monkeypatch.setenv("UMAP_LAYOUT_FAULT", "alloc")
    with pytest.raises(U.UmapLayoutError) as ei:
        U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, 10, 5)
    assert ei.value.code == U.UMAP_E_NOMEM
    monkeypatch.setenv("UMAP_LAYOUT_FAULT", "launch@3")
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, 10, 5) as h:
        with pytest.raises(U.UmapLayoutError) as ei:
            U.umap_layout_run(h, 1)
        assert ei.value.code == U.UMAP_E_DEVICE
        monkeypatch.delenv("UMAP_LAYOUT_FAULT")
        U.umap_layout_run(h, 1)
        assert np.all(np.isfinite(U.umap_layout_get(h)))
    with U.umap_layout_create(w.n, 2, r, c, v, A_DEF, B_DEF, 10, 5) as h:
        with pytest.raises(U.UmapLayoutError) as ei:
            U.umap_layout_run_epochs(h, 1, 0, 1)
        assert ei.value.code == U.UMAP_E_STATE


def test_record_overflow_redo(monkeypatch, window1m_graph):
    """A negative sample that finds its record slot full raises a flag, and the
    call's epochs are redone from the layout the call started from by the
    one-thread-per-vertex kernel: the result is the same bit for bit.  Failure
    injection gives the wavefront kernel no record slots at all."""
    w, ids, dist, (r, c, v) = window1m_graph
    E0 = synth.embedding_state(w.n, w.dim, 21, 10.0)
    case("record overflow redo, window1m, epochs 0..3 then 3..5")
    with U.umap_layout_create(w.n, w.dim, r, c, v, A_DEF, B_DEF, w.n_epochs, w.neg_rate) as h:
        assert U.umap_layout_stats(h)["table_ranges"] > 1
        U.umap_layout_set_embedding(h, E0)
        U.umap_layout_run_epochs(h, 9, 0, 3)
        st = U.umap_layout_stats(h)
        assert st["overflow_redone"] == 0
        ref3, act3 = U.umap_layout_get(h), st["active_edges"]
        U.umap_layout_run_epochs(h, 9, 3, 5)
        ref5 = U.umap_layout_get(h)

        monkeypatch.setenv("UMAP_LAYOUT_FAULT", "records")
        U.umap_layout_set_embedding(h, E0)
        U.umap_layout_run_epochs(h, 9, 0, 3)
        st = U.umap_layout_stats(h)
        assert st["overflow_redone"] == 1 and st["active_edges"] == act3
        assert np.array_equal(U.umap_layout_get(h).view(np.uint32), ref3.view(np.uint32))
        U.umap_layout_run_epochs(h, 9, 3, 5)
        assert U.umap_layout_stats(h)["overflow_redone"] == 1
        assert np.array_equal(U.umap_layout_get(h).view(np.uint32), ref5.view(np.uint32))
        monkeypatch.delenv("UMAP_LAYOUT_FAULT")
        U.umap_layout_run_epochs(h, 9, 0, 1)
        assert U.umap_layout_stats(h)["overflow_redone"] == 0


# ---------------------------------------------------------------------------
# input side: kNN lists -> B on the device
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("which", ["blobs2k", "window"])
def test_fuzzy_graph_device(which, blobs_graph):
    import torch

    if which == "blobs2k":
        w, X, ids, dist, _ = blobs_graph
        n, k = w.n, w.k
    else:
        n, k = 30011, 30
        ids, dist = synth.window_knn(n, k, synth.cluster_bounds(n, 7), seed=13)
    case(f"fuzzy graph {which}")
    di = torch.from_numpy(np.ascontiguousarray(ids)).cuda()
    dd = torch.from_numpy(np.ascontiguousarray(dist)).cuda()
    rows = torch.empty(2 * n * k, dtype=torch.int32, device="cuda")
    cols = torch.empty_like(rows)
    vals = torch.empty(2 * n * k, dtype=torch.float32, device="cuda")
    U.umap_fuzzy_graph_device(n, k, di, dd, rows, cols, vals)
    torch.cuda.synchronize()
    rg, cg, vg = rows.cpu().numpy(), cols.cpu().numpy(), vals.cpu().numpy()
    keep = (vg > 0) & (rg != cg)
    order = np.lexsort((cg[keep], rg[keep]))
    rg, cg, vg = rg[keep][order], cg[keep][order], vg[keep][order]
    ro, co, vo = O.fuzzy_union(ids, O.membership(dist, *O.smooth_knn(dist)))
    assert np.array_equal(rg, ro) and np.array_equal(cg, co)
    ulp = np.abs(vg.view(np.int32).astype(np.int64) - vo.astype(np.float32).view(np.int32).astype(np.int64))
    assert ulp.max() <= 1
    # and it ingests into the same graph as the oracle's union (up to those ulps)
    with U.umap_layout_create_device(n, 2, rows, cols, vals, 2 * n * k, A_DEF, B_DEF, 200, 5) as h:
        row_ptr, col, eps = U.umap_layout_get_graph(h)
    g = O.prep(n, ro, co, vo.astype(np.float32), 200)
    assert np.array_equal(row_ptr, g.row_ptr) and np.array_equal(col, g.col)
    assert np.allclose(eps, g.eps, rtol=1e-6, atol=0)


def test_probes():
    """The measurement probes run and the copy probe copies."""
    import torch

    case("copy and gather probes")
    src = torch.arange(1 << 16, dtype=torch.float32, device="cuda")
    dst = torch.zeros_like(src)
    U.umap_probe_copy(src, dst, src.numel() * 4)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    table = torch.ones(2 * 4096, dtype=torch.float32, device="cuda")
    out = torch.zeros(512, dtype=torch.float32, device="cuda")
    U.umap_probe_gather(table, 4096, 512, 2, out)
    torch.cuda.synchronize()
    assert float(out.abs().sum()) == 0.0


# ---------------------------------------------------------------------------
# quality: trustworthiness on the GPU (Alg. 1) against the oracle's
# ---------------------------------------------------------------------------

# a rank decided differently by fp32 than by the oracle's fp64 (a pair of input
# distances closer than fp32 resolves) moves T by 2 / (n k (2n - 3k - 1)) per unit
TW_TOL = 2e-6


@pytest.mark.parametrize("k", [5, 15, 50])
def test_trustworthiness_blobs(blobs_graph, k):
    import torch

    w, X, ids, dist, _ = blobs_graph
    rng = np.random.default_rng(k)
    for label, Y in [("pca-like", X[:, :2].copy()), ("noise", rng.normal(size=(w.n, 2)).astype(np.float32)),
                     ("3-d", (X[:, :3] + 0.5 * rng.normal(size=(w.n, 3))).astype(np.float32))]:
        case(f"trustworthiness blobs2k k={k} {label}")
        tg = U.umap_trustworthiness(torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda(), k)
        to = O.trustworthiness(X, Y, k)
        print(f"  T(gpu) = {tg:.9f}  T(oracle) = {to:.9f}  diff = {tg - to:.2e}", flush=True)
        assert abs(tg - to) <= TW_TOL


def test_trustworthiness_ragged_shapes():
    """n not a multiple of the 64-point tiles, d not a multiple of the 16-feature
    chunks, an identity embedding (T = 1), and a one-dimensional embedding."""
    import torch

    rng = np.random.default_rng(5)
    n, d = 3001, 37
    X = rng.normal(size=(n, d)).astype(np.float32)
    Xg = torch.from_numpy(X).cuda()
    case("trustworthiness identity n=3001 d=37")
    # the embedding equal to the input in a subspace it is ranked by: T = 1
    Z = np.zeros((n, 16), np.float32)
    Z[:, :16] = X[:, :16]
    X16 = np.zeros_like(X)
    X16[:, :16] = X[:, :16]
    t_id = U.umap_trustworthiness(torch.from_numpy(X16).cuda(), torch.from_numpy(Z).cuda(), 15)
    assert 1.0 - TW_TOL <= t_id <= 1.0
    for dim in (1, 2):
        case(f"trustworthiness n=3001 d=37 dim={dim}")
        Y = (X[:, :dim] + 0.2 * rng.normal(size=(n, dim))).astype(np.float32)
        tg = U.umap_trustworthiness(Xg, torch.from_numpy(Y).cuda(), 15)
        to = O.trustworthiness(X, Y, 15)
        print(f"  T(gpu) = {tg:.9f}  T(oracle) = {to:.9f}", flush=True)
        assert abs(tg - to) <= TW_TOL
    case("trustworthiness rejects a non-finite embedding")
    Y = rng.normal(size=(n, 2)).astype(np.float32)
    Y[7, 1] = np.nan
    with pytest.raises(U.UmapLayoutError) as ei:
        U.umap_trustworthiness(Xg, torch.from_numpy(Y).cuda(), 15)
    assert ei.value.code == U.UMAP_E_INVAL


def _knn_torch(X, k, batch=4096):
    """Exact Euclidean kNN (self excluded) of the rows of X with torch on the
    GPU: the input preparation of the image-like workload (its 70,000 x 784
    distance matrix is too slow for a numpy test).  Both layouts below are run
    on the same lists, so these serve as their common input."""
    import torch

    Xg = torch.from_numpy(X).cuda()
    sq = (Xg * Xg).sum(1)
    n = X.shape[0]
    ids = np.empty((n, k), np.int32)
    dist = np.empty((n, k), np.float32)
    for s in range(0, n, batch):
        t = min(n, s + batch)
        D = sq[s:t, None] + sq[None, :] - 2.0 * (Xg[s:t] @ Xg.T)
        D[torch.arange(t - s), torch.arange(s, t)] = float("inf")
        d, i = torch.topk(D, k, dim=1, largest=False, sorted=True)
        ids[s:t] = i.int().cpu().numpy()
        dist[s:t] = torch.sqrt(torch.clamp(d, min=0.0)).cpu().numpy()
    return ids, dist


def test_full_run_trustworthiness_image70k():
    """The image-like workload at full size (70,000 x 784, 10 clusters, k = 15,
    200 epochs): T@15 of the GPU layout within 0.01 of the oracle's layout, both
    scored by the GPU trustworthiness (pinned against the oracle's above)."""
    import torch

    w = synth.WORKLOADS["image70k"]
    case("image70k: points and kNN")
    X, _ = synth.workload_points(w)
    ids, dist = _knn_torch(X, w.k)
    r, c, v = O.fuzzy_graph(ids, dist)
    a, b = O.fit_ab(w.spread, w.min_dist)
    g = O.prep(w.n, r, c, v, w.n_epochs)
    seed = 3
    case("image70k: GPU layouts (synchronous, asynchronous)")
    with U.umap_layout_create(w.n, w.dim, r, c, v, a, b, w.n_epochs, w.neg_rate) as h:
        _check_graph(h, g)
        U.umap_layout_run(h, seed)
        Eg = U.umap_layout_get(h)
        st = U.umap_layout_stats(h)
        U.umap_layout_set_mode(h, U.UMAP_MODE_ASYNC)
        U.umap_layout_run(h, seed)
        Ea = U.umap_layout_get(h)
        sta = U.umap_layout_stats(h)
    case("image70k: oracle layout")
    t0 = time.perf_counter()
    Eo, act = O.run(g, w.dim, a, b, w.n_epochs, w.neg_rate, seed)
    to_s = time.perf_counter() - t0
    assert st["active_edges"] == int(act.sum()) == sta["active_edges"]
    assert np.all(np.isfinite(Eg)) and np.all(np.isfinite(Ea))
    case("image70k: trustworthiness of the three layouts")
    Xg = torch.from_numpy(X).cuda()
    tg = U.umap_trustworthiness(Xg, torch.from_numpy(Eg).cuda(), 15)
    ta = U.umap_trustworthiness(Xg, torch.from_numpy(Ea).cuda(), 15)
    to = U.umap_trustworthiness(Xg, torch.from_numpy(Eo.astype(np.float32)).cuda(), 15)
    print(f"  T@15(gpu) = {tg:.5f}  T@15(gpu async) = {ta:.5f}  T@15(oracle) = {to:.5f}; GPU epochs "
          f"{st['epochs_ms']:.2f} ms ({st['edge_updates'] / (st['epochs_ms'] * 1e-3):.3e} edge-updates/s), "
          f"oracle run {to_s:.2f} s on {O.num_threads()} threads", flush=True)
    assert abs(tg - to) <= 0.01
    assert abs(ta - to) <= 0.01
