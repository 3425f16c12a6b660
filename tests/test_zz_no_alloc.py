"""The no-allocation fuzzy-graph entry point (umap_fuzzy_graph_device_noalloc:
scratch in a static per-GPU array) against the allocating one, through the C
ABI: bit-identical rows, cols and vals on two calls in a row, the second with
a smaller input (the array keeps the first call's contents), and the size
limit rejected with UMAP_E_INVAL."""

import sys

import numpy as np
import pytest

from paper_2008_00325_amd import synth
from paper_2008_00325_amd import umap_layout as U

pytestmark = pytest.mark.gpu


def case(msg):
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def _graph(entry, n, k, di, dd):
    import torch

    rows = torch.full((2 * n * k,), -7, dtype=torch.int32, device="cuda")
    cols = torch.full_like(rows, -7)
    vals = torch.full((2 * n * k,), -7.0, dtype=torch.float32, device="cuda")
    entry(n, k, di, dd, rows, cols, vals)
    torch.cuda.synchronize()
    return rows.cpu().numpy(), cols.cpu().numpy(), vals.cpu().numpy()


def test_no_alloc_equals_allocating_entry_point():
    import torch

    torch.cuda.init()
    torch.cuda.set_device(0)
    for n, k, clusters, seed in [(200_003, 30, 11, 21), (4_099, 15, 3, 22)]:
        ids, dist = synth.window_knn(n, k, synth.cluster_bounds(n, clusters), seed=seed)
        # zero distances in some rows: rho = 0 and sigma on its floor
        dist[np.random.default_rng(seed).random(n) < 0.03] = 0.0
        dist = np.sort(dist, axis=1)
        di = torch.from_numpy(np.ascontiguousarray(ids)).cuda()
        dd = torch.from_numpy(np.ascontiguousarray(dist)).cuda()
        case(f"no-alloc fuzzy graph n={n} k={k}")
        want = _graph(U.umap_fuzzy_graph_device, n, k, di, dd)
        got = _graph(U.umap_fuzzy_graph_device_noalloc, n, k, di, dd)
        assert np.array_equal(got[0], want[0])
        assert np.array_equal(got[1], want[1])
        assert np.array_equal(got[2].view(np.int32), want[2].view(np.int32))
        assert (got[2] > 0).sum() >= n * k   # every forward slot holds a membership
    case("no-alloc fuzzy graph size limit")
    p = torch.zeros(16, dtype=torch.int32, device="cuda").data_ptr()
    L = U.lib()
    assert L.umap_fuzzy_graph_device_noalloc(2**20 + 1, 1, p, p, p, p, p, None) == U.UMAP_E_INVAL
    # an id out of range is reported, and the next call is clean again
    ids = np.zeros((64, 3), np.int32)
    ids[5, 1] = 64
    dist = np.ones((64, 3), np.float32)
    di = torch.from_numpy(ids).cuda()
    dd = torch.from_numpy(dist).cuda()
    with pytest.raises(U.UmapLayoutError) as ei:
        _graph(U.umap_fuzzy_graph_device_noalloc, 64, 3, di, dd)
    assert ei.value.code == U.UMAP_E_INVAL
    ids[5, 1] = 6
    di = torch.from_numpy(ids).cuda()
    got = _graph(U.umap_fuzzy_graph_device_noalloc, 64, 3, di, dd)
    want = _graph(U.umap_fuzzy_graph_device, 64, 3, di, dd)
    assert np.array_equal(got[2].view(np.int32), want[2].view(np.int32))
