"""Pins of the oracle's random streams (Philox4x32-10, Salmon et al., SC'11).

The generator is not described in the paper (it only says a user seed controls
the random state, reproducibility section); the oracle adopts Philox4x32-10.
It is pinned against an independent implementation of the same published
generator -- PyTorch's header-only ``at::philox_engine`` compiled here with g++
-- and by distribution checks of the derived quantities.
"""

import os
import subprocess
import sysconfig

import numpy as np
import pytest

_REF_SRC = r"""
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
#include <cstdint>
// stdin: lines "seed c0 c1 c2 c3"; stdout: the four output words
int main() {
  unsigned long long seed; unsigned c0, c1, c2, c3;
  while (std::scanf("%llu %u %u %u %u", &seed, &c0, &c1, &c2, &c3) == 5) {
    uint64_t offset = (uint64_t)c0 | ((uint64_t)c1 << 32);
    uint64_t subseq = (uint64_t)c2 | ((uint64_t)c3 << 32);
    at::philox_engine eng(seed, subseq, offset);
    unsigned w0 = eng(), w1 = eng(), w2 = eng(), w3 = eng();
    std::printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
"""


def _torch_include():
    import torch

    return os.path.join(os.path.dirname(torch.__file__), "include")


@pytest.fixture(scope="module")
def torch_philox(tmp_path_factory):
    d = tmp_path_factory.mktemp("philox")
    src = d / "ref.cpp"
    src.write_text(_REF_SRC)
    exe = d / "ref"
    r = subprocess.run(["g++", "-std=c++17", "-O1", "-I", _torch_include(), str(src), "-o", str(exe)],
                       capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("cannot build the torch Philox reference: " + r.stderr[-400:])

    def run(seeds, ctrs):
        inp = "\n".join(f"{int(s)} {c[0]} {c[1]} {c[2]} {c[3]}" for s, c in zip(seeds, ctrs)) + "\n"
        out = subprocess.run([str(exe)], input=inp, capture_output=True, text=True, check=True).stdout
        return np.array([[int(w) for w in line.split()] for line in out.strip().splitlines()], dtype=np.uint32)

    return run


def test_philox_matches_independent_implementation(orc, torch_philox):
    rng = np.random.default_rng(11)
    m = 4000
    seeds = rng.integers(0, 2**63, m, dtype=np.uint64)
    seeds[:4] = [0, 1, 2**32, 2**64 - 1]
    ctrs = rng.integers(0, 2**32, (m, 4), dtype=np.uint64).astype(np.uint32)
    ctrs[0] = 0
    ctrs[1] = 0xFFFFFFFF
    ref = torch_philox(seeds, ctrs)
    got = np.stack([orc.philox4x32_10(ctrs[t:t + 1], (int(seeds[t]) & 0xFFFFFFFF, int(seeds[t]) >> 32))[0]
                    for t in range(m)])
    assert np.array_equal(got, ref)


def test_negative_and_init_words_follow_the_stream_layout(orc):
    seed = 0x0123456789ABCDEF
    key = (seed & 0xFFFFFFFF, seed >> 32)
    n = 1_000_003
    e, ep = 5_000_000_123, 17
    ks = orc.negative_vertices(seed, ep, e, 1, 7, n)[0]
    for r in range(7):
        ctr = np.array([[e & 0xFFFFFFFF, e >> 32, ep, 0x4E470000 | (r >> 2)]], dtype=np.uint32)
        u = int(orc.philox4x32_10(ctr, key)[0, r & 3])
        assert ks[r] == (u * n) >> 32
    E = orc.init_layout(3, 6, seed)
    for i in range(3):
        for d in range(6):
            ctr = np.array([[i, 0, d >> 2, 0x494E0000]], dtype=np.uint32)
            u = int(orc.philox4x32_10(ctr, key)[0, d & 3])
            unit = np.float32(((u >> 8) - (1 << 23)) * 2.0**-23)
            assert E[i, d] == np.float32(unit * np.float32(10.0))


def test_negative_vertices_uniform(orc):
    n = 1000
    ks = orc.negative_vertices(7, 3, 0, 200_000, 5, n).ravel()
    assert ks.max() < n
    counts = np.bincount(ks, minlength=n)
    expect = ks.size / n
    chi2 = float(((counts - expect) ** 2 / expect).sum())
    # 999 degrees of freedom: mean 999, sd ~44.7; accept within 5 sd
    assert abs(chi2 - (n - 1)) < 5 * np.sqrt(2 * (n - 1))
    # different epochs, edges and seeds give different draws
    a = orc.negative_vertices(7, 3, 0, 1000, 5, n)
    assert not np.array_equal(a, orc.negative_vertices(7, 4, 0, 1000, 5, n))
    assert not np.array_equal(a, orc.negative_vertices(8, 3, 0, 1000, 5, n))
    assert not np.array_equal(a, orc.negative_vertices(7, 3, 1, 1000, 5, n))


def test_init_uniform_range(orc):
    E = orc.init_layout(100_000, 2, 3)
    assert E.min() >= -10.0 and E.max() < 10.0
    # values lie on the 10 * 2^-23 grid of the 24-bit construction
    q = E.astype(np.float64) / 10.0 * 2**23
    assert np.allclose(q, np.round(q), atol=1e-3)
    h, _ = np.histogram(E.ravel(), bins=20, range=(-10, 10))
    assert abs(h / h.mean() - 1).max() < 0.05
    assert abs(E.mean()) < 0.05
