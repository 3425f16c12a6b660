"""Writes window_quality.json: the oracle's full runs of the graph-only
workloads (1M vertices k = 15 in 2-D, 1M vertices k = 30 in 3-D, 5M vertices
k = 15 in 2-D; 200 epochs, 5 negatives, min_dist 0.1, spread 1) scored on a
seeded sample of 10,000 vertices by recall@15 of the input neighbours and the
objective of the UMAP section.  The layout of a graph-only workload has no
input coordinates, so these two measures stand in for trustworthiness.

Calls only the oracle and the seeded input generators.  Usage (from the
repository root):  python tests/golden/make_window_quality.py [workload ...]
It takes about 5 minutes per million vertices on 8 cores.
"""

import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle as O  # noqa: E402
from paper_2008_00325_amd import synth  # noqa: E402

OUT = os.path.join(HERE, "window_quality.json")
SEED = 1
NAMES = ["window1m", "window1m_k30", "window5m"]


def score(w, ids, g, E, a, b):
    rows, neg = synth.quality_sample(w.n)
    return {
        "recall15": O.recall_at_k(ids, E, rows, 15),
        "objective": O.objective(g, E, a, b, w.neg_rate, rows, neg),
    }


def main(names):
    doc = json.load(open(OUT)) if os.path.exists(OUT) else {}
    doc["citation"] = (
        "Oracle full runs (epoch-synchronous fp64 layout SGD of the UMAP section, embedding-updates section) "
        "of the graph-only workloads; recall@15 of the first 15 input neighbours among the 15 nearest "
        "layout neighbours, and the cross-entropy objective of the UMAP section restricted to the edges of "
        "the sampled vertices (edge term weighted by its sampling frequency 1/eps, negatives fixed per "
        "vertex).  Sample: synth.quality_sample(n) (10,000 vertices, 64 negatives each, seed 12345).")
    doc["seed"] = SEED
    for name in names:
        w = synth.WORKLOADS[name]
        t0 = time.time()
        ids, dist = synth.workload_knn(w)
        r, c, v = O.fuzzy_graph(ids, dist)
        g = O.prep(w.n, r, c, v, w.n_epochs)
        del r, c, v
        a, b = O.fit_ab(w.spread, w.min_dist)
        t1 = time.time()
        E, act = O.run(g, w.dim, a, b, w.n_epochs, w.neg_rate, SEED)
        t2 = time.time()
        entry = score(w, ids, g, E, a, b)
        init = score(w, ids, g, O.init_layout(w.n, w.dim, SEED), a, b)
        entry.update({
            "recall15_init": init["recall15"],
            "objective_init": init["objective"],
            "active_edges": int(act.sum()),
            "oracle_run_seconds": round(t2 - t1, 1),
            "oracle_threads": O.num_threads(),
        })
        doc[name] = entry
        print(f"{name}: graph {t1 - t0:.0f} s, run {t2 - t1:.0f} s, {entry}", flush=True)
        with open(OUT, "w") as f:
            json.dump(doc, f, indent=1)
            f.write("\n")


if __name__ == "__main__":
    main(sys.argv[1:] or NAMES)
