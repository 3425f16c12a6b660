"""Single-epoch parity on 40 seeded random cases: a random symmetric graph
(n from 1 to 5,000, mean degree 0 to 40), random embedding dimension (1-16),
neg_rate (0-12), epoch count and epoch, a random fp32 state; both epoch
kernels against the oracle (max |GPU - oracle| <= 1e-4, exact sampled-edge
count).  The cases are drawn once from a fixed seed, so a failure names a
case that can be rerun."""

import sys

import numpy as np
import pytest

import oracle as O
from paper_2008_00325_amd import synth
from paper_2008_00325_amd import umap_layout as U

pytestmark = pytest.mark.gpu

TOL = 1e-4
A_DEF, B_DEF = 1.5769434, 0.8950608


def _cases(count=40, seed=2024):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(count):
        n = int(rng.choice([1, 2, 3, 17, 64, 65, 129, 500, 1000, 2047, 3001, 5000]))
        deg = int(rng.integers(0, 41))
        dim = int(rng.integers(1, 17))
        R = int(rng.integers(0, 13))
        N = int(rng.choice([1, 2, 7, 50, 200, 500]))
        ep = int(rng.integers(0, N))
        out.append((c, n, deg, dim, R, N, ep, int(rng.integers(0, 2**31))))
    return out


@pytest.fixture(scope="module", autouse=True)
def torch_device_first():
    import torch

    torch.cuda.init()
    torch.cuda.set_device(0)


@pytest.mark.parametrize("case", _cases(), ids=lambda c: f"case{c[0]}-n{c[1]}-deg{c[2]}-dim{c[3]}-R{c[4]}-N{c[5]}")
def test_random_case(case):
    c, n, deg, dim, R, N, ep, seed = case
    print(f"[gpu case] random case {c}: n {n} deg {deg} dim {dim} R {R} N {N} epoch {ep} seed {seed}", flush=True)
    sys.stdout.flush()
    if deg > 0 and n > 1:
        r, col, v = synth.random_symmetric_coo(n, deg, seed % 100000)
    else:
        r = col = np.zeros(0, np.int32)
        v = np.zeros(0, np.float32)
    g = O.prep(n, r, col, v, N)
    E = synth.embedding_state(n, dim, seed % 1000, 10.0)
    ref, act = O.epoch(g, E, ep, A_DEF, B_DEF, N, R, seed)
    outs = []
    with U.umap_layout_create(n, dim, r, col, v, A_DEF, B_DEF, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, seed, ep, ep + 1)
            got = U.umap_layout_get(h)
            outs.append(got)
            err = float(np.abs(got.astype(np.float64) - ref).max()) if n * dim else 0.0
            st = U.umap_layout_stats(h)
            assert err <= TOL, (kernel, err)
            assert st["active_edges"] == act and st["overflow_redone"] == 0
    # the terms are summed as exact integers, so the wave kernels and the
    # one-thread-per-vertex kernel give the same bits
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


def _transform_cases(count=12, seed=77):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(count):
        n_table = int(rng.choice([130, 500, 4096, 20000, 300000]))
        n_new = int(rng.choice([1, 2, 63, 64, 1000, 7777]))
        k = int(rng.integers(1, 31))
        dim = int(rng.integers(1, 17))
        R = int(rng.integers(0, 13))
        N = int(rng.choice([1, 3, 50, 100]))
        out.append((c, n_table, n_new, k, dim, R, N, int(rng.integers(0, N)), int(rng.integers(0, 2**31))))
    return out


@pytest.mark.parametrize("case", _transform_cases(),
                         ids=lambda c: f"t{c[0]}-table{c[1]}-new{c[2]}-k{c[3]}-dim{c[4]}-R{c[5]}-N{c[6]}")
def test_random_transform_case(case):
    """A transform: new points with k scattered edges each into a random
    frozen table (both kernels)."""
    c, n_table, n_new, k, dim, R, N, ep, seed = case
    print(f"[gpu case] random transform {c}: table {n_table} new {n_new} k {k} dim {dim} R {R} N {N} epoch {ep}",
          flush=True)
    rng = np.random.default_rng(seed)
    k = min(k, n_table)
    rows = np.repeat(np.arange(n_new, dtype=np.int32), k)
    cols = np.concatenate([rng.choice(n_table, size=k, replace=False) for _ in range(n_new)]).astype(np.int32)
    vals = rng.uniform(0.01, 1.0, size=rows.size).astype(np.float32)
    T = synth.embedding_state(n_table, dim, seed % 1000, 10.0)
    Y = synth.embedding_state(n_new, dim, seed % 997, 10.0)
    g = O.prep_bipartite(n_new, n_table, rows, cols, vals, N)
    a, b = A_DEF, B_DEF
    with U.umap_transform_create(n_new, T, rows, cols, vals, a, b, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_embedding(h, Y)
            U.umap_layout_run_epochs(h, seed, ep, ep + 1)
            ref, act = O.frozen_epoch(g, Y, T, ep, a, b, N, R, seed)
            err = float(np.abs(U.umap_layout_get(h).astype(np.float64) - ref).max())
            st = U.umap_layout_stats(h)
            assert err <= TOL, (kernel, err)
            assert st["active_edges"] == act and st["overflow_redone"] == 0


@pytest.mark.parametrize("case", _cases(12, seed=99), ids=lambda c: f"rows{c[0]}-n{c[1]}-dim{c[3]}-R{c[4]}")
def test_random_row_range_case(case):
    """A random row range of a random graph: its rows bit-identical to the
    whole epoch's, the others unchanged, both within 1e-4 of the oracle."""
    c, n, deg, dim, R, N, ep, seed = case
    rng = np.random.default_rng(seed)
    r0 = int(rng.integers(0, n))
    r1 = int(rng.integers(r0 + 1, n + 1))
    print(f"[gpu case] random rows {c}: n {n} rows [{r0}, {r1}) deg {deg} dim {dim} R {R} N {N} epoch {ep}",
          flush=True)
    if deg > 0 and n > 1:
        r, col, v = synth.random_symmetric_coo(n, deg, seed % 100000)
    else:
        r = col = np.zeros(0, np.int32)
        v = np.zeros(0, np.float32)
    g = O.prep(n, r, col, v, N)
    E = synth.embedding_state(n, dim, seed % 1000, 10.0)
    with U.umap_layout_create(n, dim, r, col, v, A_DEF, B_DEF, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_rows(h, 0, n)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, seed, ep, ep + 1)
            full = U.umap_layout_get(h)
            U.umap_layout_set_rows(h, r0, r1)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, seed, ep, ep + 1)
            got = U.umap_layout_get(h)
            assert np.array_equal(got[r0:r1].view(np.uint32), full[r0:r1].view(np.uint32))
            assert np.array_equal(got[:r0].view(np.uint32), E[:r0].view(np.uint32))
            assert np.array_equal(got[r1:].view(np.uint32), E[r1:].view(np.uint32))
            delta = O.epoch_rows(g, E, ep, A_DEF, B_DEF, N, R, seed, np.arange(r0, r1, dtype=np.int64))
            ref = E[r0:r1].astype(np.float64) + delta
            assert float(np.abs(got[r0:r1].astype(np.float64) - ref).max()) <= TOL


def _graph_cases(count=8, seed=5150):
    rng = np.random.default_rng(seed)
    return [(c, int(rng.choice([2, 17, 300, 4000, 20000])), int(rng.integers(1, 65)), int(rng.integers(0, 2**31)))
            for c in range(count)]


@pytest.mark.parametrize("case", _graph_cases(), ids=lambda c: f"g{c[0]}-n{c[1]}-k{c[2]}")
def test_random_fuzzy_graph_case(case):
    """The device fuzzy graph on random kNN lists with the awkward rows: a
    leading run of zero distances (rho from the first positive one), all-zero
    rows (sigma floored from the global mean), repeated distances, self ids
    in some lists (ignored): structure identical to the oracle's union, values
    within one fp32 ulp."""
    import torch

    c, n, k, seed = case
    k = min(k, n - 1) if n > 1 else 1
    print(f"[gpu case] random fuzzy graph {c}: n {n} k {k}", flush=True)
    rng = np.random.default_rng(seed)
    ids = np.empty((n, k), np.int32)
    for i in range(n):
        ids[i] = rng.choice(n, size=k, replace=False)
    dist = np.sort(rng.exponential(1.0, size=(n, k)), axis=1).astype(np.float32)
    dist = np.round(dist, 1)                                   # repeated values
    zero_lead = rng.random(n) < 0.2
    dist[zero_lead, : max(1, k // 3)] = 0.0
    dist[rng.random(n) < 0.05] = 0.0                           # whole rows at distance 0
    dist = np.sort(dist, axis=1)
    di = torch.from_numpy(ids).cuda()
    dd = torch.from_numpy(dist).cuda()
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
    vo = vo.astype(np.float32)
    ko = (vo > 0) & (ro != co)
    ro, co, vo = ro[ko], co[ko], vo[ko]
    # rows whose sigma sits on its floor have memberships that underflow; a
    # value at the edge of fp32's range may be 0 on one side only
    gpu = dict(zip(zip(rg.tolist(), cg.tolist()), vg.tolist()))
    ora = dict(zip(zip(ro.tolist(), co.tolist()), vo.tolist()))
    for key in set(gpu) ^ set(ora):
        assert gpu.get(key, ora.get(key)) < 1e-30, key
    both = sorted(set(gpu) & set(ora))
    a = np.array([gpu[x] for x in both], np.float32)
    b = np.array([ora[x] for x in both], np.float32)
    big = (a >= 1e-30) | (b >= 1e-30)
    ulp = np.abs(a.view(np.int32).astype(np.int64) - b.view(np.int32).astype(np.int64))
    assert ulp[big].max(initial=0) <= 1
    assert len(both) > 0.9 * len(ora)


def _trust_cases(count=10, seed=31337):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(count):
        n = int(rng.choice([1000, 2047, 3001, 5000]))
        k = int(rng.integers(1, 65))
        while 2 * n - 3 * k - 1 <= 0:
            k //= 2
        out.append((c, n, int(rng.integers(1, 101)), int(rng.integers(1, 17)), max(k, 1), int(rng.integers(0, 2**31))))
    return out


@pytest.mark.parametrize("case", _trust_cases(), ids=lambda c: f"tw{c[0]}-n{c[1]}-d{c[2]}-dim{c[3]}-k{c[4]}")
def test_random_trustworthiness_case(case):
    """GPU trustworthiness against the oracle's on random shapes: every rank
    kernel instance (k up to 64), feature counts that are not multiples of 4,
    embeddings of 1-16 components.  The GPU ranks by fp32 distances (matrix
    tiles), the oracle by fp64 ones, so a near-tie may be ordered differently;
    each such swap moves T by 2 / (n k (2n - 3k - 1)), under 2e-8 for n >= 1000
    (at n = 129, k = 52 one swap alone is 2.95e-6), so the sizes here keep the
    2e-6 bound many swaps wide."""
    import torch

    c, n, d, dim, k, seed = case
    print(f"[gpu case] random trustworthiness {c}: n {n} d {d} dim {dim} k {k}", flush=True)
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    Y = rng.standard_normal((n, dim)).astype(np.float32)
    got = U.umap_trustworthiness(torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda(), k)
    ref = O.trustworthiness(X, Y, k)
    assert abs(got - ref) <= 2e-6, (got, ref)
