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
    with U.umap_layout_create(n, dim, r, col, v, A_DEF, B_DEF, N, R) as h:
        for kernel in (0, 1):
            U.umap_layout_set_kernel(h, kernel)
            U.umap_layout_set_embedding(h, E)
            U.umap_layout_run_epochs(h, seed, ep, ep + 1)
            ref, act = O.epoch(g, E, ep, A_DEF, B_DEF, N, R, seed)
            got = U.umap_layout_get(h)
            err = float(np.abs(got.astype(np.float64) - ref).max()) if n * dim else 0.0
            st = U.umap_layout_stats(h)
            assert err <= TOL, (kernel, err)
            assert st["active_edges"] == act and st["overflow_redone"] == 0
