"""One GPU's share of a row-sharded layout (umap_layout_set_rows), through the
C ABI:
  * each row of a range is bit-identical to the same row of an epoch over all
    rows from the same layout, and the rows outside keep their values, so the
    shards of a split assemble the full epoch bit for bit (both kernels, the
    1M-vertex workload in the benchmark's launch configuration);
  * one epoch of a range against the oracle's update of those rows (the push
    form restricted to them): max |GPU - oracle| <= 1e-4;
  * ragged and one-row ranges, several epochs in one call, the redo path,
    a transform's new points, and the argument checks.
"""

import sys

import numpy as np
import pytest

import oracle as O
from paper_2008_00325_amd import synth
from paper_2008_00325_amd import umap_layout as U

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def torch_device_first():
    """Initialise torch's HIP runtime before the library's."""
    import torch

    torch.cuda.init()
    torch.cuda.set_device(0)


def case(msg):
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def shard_bounds(row_ptr, parts):
    """Row bounds of `parts` contiguous ranges with about equal kept edges."""
    nnz = int(row_ptr[-1])
    b = np.searchsorted(row_ptr, (np.arange(parts + 1, dtype=np.int64) * nnz) // parts, side="left")
    b[0], b[-1] = 0, row_ptr.size - 1
    return [int(x) for x in b]


def _bits(x):
    return np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)


def _shard_epoch(h, E, r0, r1, ep, seed):
    U.umap_layout_set_rows(h, r0, r1)
    U.umap_layout_set_embedding(h, E)
    U.umap_layout_run_epochs(h, seed, ep, ep + 1)
    return U.umap_layout_get(h), U.umap_layout_stats(h)


def _oracle_rows(g, E, r0, r1, ep, a, b, N, R, seed):
    delta = O.epoch_rows(g, E, ep, a, b, N, R, seed, np.arange(r0, r1, dtype=np.int64))
    return E[r0:r1].astype(np.float64) + delta


@pytest.fixture(scope="module")
def window1m():
    w = synth.WORKLOADS["window1m"]
    ids, dist = synth.workload_knn(w)
    r, c, v = O.fuzzy_graph(ids, dist)
    del ids, dist
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    return w, (r, c, v), g, a, b


def test_eight_shards_assemble_the_full_epoch_window1m(window1m):
    """The 1M-vertex, k = 15, 2-D workload split into 8 ranges of equal edges."""
    import torch

    w, (r, c, v), g, a, b = window1m
    bounds = shard_bounds(g.row_ptr, 8)
    E = synth.embedding_state(w.n, w.dim, 3, 10.0)
    dr, dc, dv = (torch.from_numpy(x).cuda() for x in (r, c, v))
    with U.umap_layout_create_device(w.n, w.dim, dr, dc, dv, r.size, a, b, w.n_epochs, w.neg_rate) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for ep in (0, w.n_epochs // 2):
                case(f"window1m kernel {kernel} epoch {ep}: full epoch")
                U.umap_layout_set_rows(h, 0, w.n)
                U.umap_layout_set_embedding(h, E)
                U.umap_layout_run_epochs(h, 11, ep, ep + 1)
                full = U.umap_layout_get(h)
                full_active = U.umap_layout_stats(h)["active_edges"]
                assembled = np.empty_like(full)
                active = 0
                for s in range(8):
                    r0, r1 = bounds[s], bounds[s + 1]
                    case(f"window1m kernel {kernel} epoch {ep}: shard {s} rows [{r0}, {r1})")
                    got, st = _shard_epoch(h, E, r0, r1, ep, 11)
                    assert st["row_first"] == r0 and st["row_last"] == r1 and st["overflow_redone"] == 0
                    assert np.array_equal(_bits(got[:r0]), _bits(E[:r0]))
                    assert np.array_equal(_bits(got[r1:]), _bits(E[r1:]))
                    assembled[r0:r1] = got[r0:r1]
                    e0, e1 = g.row_ptr[r0], g.row_ptr[r1]
                    assert st["active_edges"] == int(O.active_mask(g.eps[e0:e1], ep).sum())
                    active += st["active_edges"]
                    if s == 3:
                        ref = _oracle_rows(g, E, r0, r1, ep, a, b, w.n_epochs, w.neg_rate, 11)
                        err = float(np.abs(got[r0:r1].astype(np.float64) - ref).max())
                        print(f"  shard {s} vs oracle: max|diff| = {err:.3e}", flush=True)
                        assert err <= TOL
                assert np.array_equal(_bits(assembled), _bits(full))
                assert active == full_active


@pytest.fixture(scope="module")
def blobs():
    w = synth.WORKLOADS["blobs2k"]
    X, _ = synth.workload_points(w)
    ids, dist = O.exact_knn(X, w.k)
    r, c, v = O.fuzzy_graph(ids, dist)
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    return w, (r, c, v), g, a, b


@pytest.mark.parametrize("r0,r1", [(0, 1), (1999, 2000), (17, 1234), (0, 2000), (1000, 1001)])
def test_ragged_ranges_blobs(blobs, r0, r1):
    w, (r, c, v), g, a, b = blobs
    N, R = w.n_epochs, w.neg_rate
    E = O.init_layout(w.n, 2, 7)
    with U.umap_layout_create(w.n, 2, r, c, v, a, b, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for ep in (0, 1, N // 2, N - 1):
                case(f"blobs2k rows [{r0}, {r1}) kernel {kernel} epoch {ep}")
                U.umap_layout_set_rows(h, 0, w.n)
                U.umap_layout_set_embedding(h, E)
                U.umap_layout_run_epochs(h, 7, ep, ep + 1)
                full = U.umap_layout_get(h)
                got, st = _shard_epoch(h, E, r0, r1, ep, 7)
                assert np.array_equal(_bits(got[r0:r1]), _bits(full[r0:r1]))
                assert np.array_equal(_bits(got[:r0]), _bits(E[:r0]))
                assert np.array_equal(_bits(got[r1:]), _bits(E[r1:]))
                ref = _oracle_rows(g, E, r0, r1, ep, a, b, N, R, 7)
                assert float(np.abs(got[r0:r1].astype(np.float64) - ref).max()) <= TOL
                e0, e1 = g.row_ptr[r0], g.row_ptr[r1]
                assert st["active_edges"] == int(O.active_mask(g.eps[e0:e1], ep).sum())


def test_range_over_several_epochs(blobs):
    """Ten epochs in one call equal ten one-epoch calls; every epoch of the
    range matches the oracle fed the same state; rows outside never change;
    a run (init + epochs) with a range initialises every row."""
    w, (r, c, v), _, a, b = blobs
    N, R, seed = 40, 5, 3
    g = O.prep(w.n, r, c, v, N)     # the schedule of a 40-epoch run
    r0, r1 = 523, 1481
    E0 = O.init_layout(w.n, 2, seed)
    with U.umap_layout_create(w.n, 2, r, c, v, a, b, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_rows(h, r0, r1)
            case(f"blobs2k rows [{r0}, {r1}) kernel {kernel}: epochs 0..10 in one call")
            U.umap_layout_set_embedding(h, E0)
            U.umap_layout_run_epochs(h, seed, 0, 10)
            one_call = U.umap_layout_get(h)
            E = E0
            U.umap_layout_set_embedding(h, E)
            for ep in range(10):
                U.umap_layout_run_epochs(h, seed, ep, ep + 1)
                nxt = U.umap_layout_get(h)
                ref = _oracle_rows(g, E, r0, r1, ep, a, b, N, R, seed)
                assert float(np.abs(nxt[r0:r1].astype(np.float64) - ref).max()) <= TOL
                E = nxt
            assert np.array_equal(_bits(E), _bits(one_call))
            assert np.array_equal(_bits(E[:r0]), _bits(E0[:r0]))
            assert np.array_equal(_bits(E[r1:]), _bits(E0[r1:]))
            case(f"blobs2k rows [{r0}, {r1}) kernel {kernel}: run")
            U.umap_layout_run(h, seed)
            out = U.umap_layout_get(h)
            assert np.array_equal(_bits(out[:r0]), _bits(E0[:r0]))
            assert np.array_equal(_bits(out[r1:]), _bits(E0[r1:]))
            assert np.all(np.isfinite(out))


def test_range_redo_path(monkeypatch, window1m):
    """With no record slots, the range's epochs are redone by the
    one-thread-per-vertex kernel over the same rows: same result bit for bit."""
    w, (r, c, v), g, a, b = window1m
    bounds = shard_bounds(g.row_ptr, 8)
    r0, r1 = bounds[5], bounds[6]
    E = synth.embedding_state(w.n, w.dim, 8, 10.0)
    with U.umap_layout_create(w.n, w.dim, r, c, v, a, b, w.n_epochs, w.neg_rate) as h:
        U.umap_layout_set_rows(h, r0, r1)
        case(f"window1m rows [{r0}, {r1}): epochs 4..6")
        U.umap_layout_set_embedding(h, E)
        U.umap_layout_run_epochs(h, 2, 4, 6)
        ref = U.umap_layout_get(h)
        assert U.umap_layout_stats(h)["overflow_redone"] == 0
        monkeypatch.setenv("UMAP_LAYOUT_FAULT", "records")
        case(f"window1m rows [{r0}, {r1}): epochs 4..6, no record slots")
        U.umap_layout_set_embedding(h, E)
        U.umap_layout_run_epochs(h, 2, 4, 6)
        assert U.umap_layout_stats(h)["overflow_redone"] == 1
        assert np.array_equal(_bits(U.umap_layout_get(h)), _bits(ref))
        monkeypatch.delenv("UMAP_LAYOUT_FAULT")


def test_transform_new_points_in_ranges():
    """A transform's new points split in three ranges assemble its full epoch."""
    n_table, n_new, N, R = 5000, 3000, 100, 5
    rows, cols, vals = synth.transform_graph(n_new, n_table, k=15, seed=6)
    T = synth.embedding_state(n_table, 2, 9, 10.0)
    Y = synth.embedding_state(n_new, 2, 10, 10.0)
    gb = O.prep_bipartite(n_new, n_table, rows, cols, vals, N)
    a, b = O.fit_ab(1.0, 0.1)
    with U.umap_transform_create(n_new, T, rows, cols, vals, a, b, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            for ep in (0, N // 2):
                case(f"transform kernel {kernel} epoch {ep}")
                U.umap_layout_set_rows(h, 0, n_new)
                U.umap_layout_set_embedding(h, Y)
                U.umap_layout_run_epochs(h, 4, ep, ep + 1)
                full = U.umap_layout_get(h)
                ref, _ = O.frozen_epoch(gb, Y, T, ep, a, b, N, R, 4)
                assert float(np.abs(full.astype(np.float64) - ref).max()) <= TOL
                assembled = np.empty_like(full)
                for r0, r1 in ((0, 1111), (1111, 1112), (1112, n_new)):
                    got, _ = _shard_epoch(h, Y, r0, r1, ep, 4)
                    assert np.array_equal(_bits(got[:r0]), _bits(Y[:r0]))
                    assert np.array_equal(_bits(got[r1:]), _bits(Y[r1:]))
                    assembled[r0:r1] = got[r0:r1]
                assert np.array_equal(_bits(assembled), _bits(full))


def test_range_argument_checks(blobs):
    w, (r, c, v), g, a, b = blobs
    with U.umap_layout_create(w.n, 2, r, c, v, a, b, 10, 5) as h:
        for r0, r1 in ((-1, 5), (5, 5), (6, 5), (0, w.n + 1)):
            with pytest.raises(U.UmapLayoutError) as ei:
                U.umap_layout_set_rows(h, r0, r1)
            assert ei.value.code == U.UMAP_E_INVAL
        st = U.umap_layout_stats(h)
        assert (st["row_first"], st["row_last"]) == (0, w.n)
        U.umap_layout_set_rows(h, 10, 20)
        U.umap_layout_set_mode(h, U.UMAP_MODE_ASYNC)
        U.umap_layout_set_embedding(h, O.init_layout(w.n, 2, 1))
        with pytest.raises(U.UmapLayoutError) as ei:
            U.umap_layout_run_epochs(h, 1, 0, 1)
        assert ei.value.code == U.UMAP_E_INVAL and "set_rows" in U.umap_layout_last_error()
        U.umap_layout_set_rows(h, 0, w.n)
        U.umap_layout_run_epochs(h, 1, 0, 1)
        assert np.all(np.isfinite(U.umap_layout_get(h)))
