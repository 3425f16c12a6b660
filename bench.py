"""Benchmark of the MI355X layout SGD (one GPU).

One step = one pass of the whole layout path over the resident graph B of the
1M-vertex workload (k = 15 window kNN, 2-D, 200 epochs, 5 negatives per
sampled edge): device ingest (drop / prune / sort / CSR / eps / symmetry
check), random initialisation, the 200 epoch kernels and the device-to-device
copy of the result.  B is built on the GPU from the seeded kNN lists before the
timed region.

value = edge-updates (sampled edges + drawn negatives, over all epochs of all
timed steps) / wall time of the timed steps.  The 200-epoch layout time, the
ingest time and the epoch kernel's roofline come from the library's HIP events
on the stream the kernels run on.  The CPU baseline times the C oracle on a
bounded sample of epochs of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
Prints one JSON line on stdout.
"""

from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import re
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
# L2 request rate of the chip: 8 XCDs x 16 L2 channels, one 128-byte request per channel per clock at 2.4 GHz
L2_REQUEST_PEAK_G_PER_S = 8 * 16 * 2.4
# HBM traffic of one epoch from rocprofv3 FETCH_SIZE / WRITE_SIZE passes (scaled by the
# same counters on the library's copy probe); valid while the kernel sources hash the same
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "epoch_window1m.md")
KERNEL_SOURCES = ["paper_2008_00325_amd/csrc/kernels_layout.hip", "paper_2008_00325_amd/csrc/layout_device.hpp",
                  "paper_2008_00325_amd/csrc/internal.hpp"]


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_hash() -> str:
    """Hash of the epoch kernels' code with comments and whitespace removed, so
    that an edit of the comments keeps the recorded profile valid."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def profiled_traffic(workload: str):
    """Bytes per epoch recorded in the profile summary, if it was taken on the
    current kernel sources and this workload; else None."""
    if not os.path.exists(PROFILE_TRAFFIC):
        return None
    fields = {}
    with open(PROFILE_TRAFFIC) as f:
        for line in f:
            m = re.match(r"^- (kernel_hash|workload|traffic_bytes_per_epoch): `?([^`\s]+)`?", line.strip())
            if m:
                fields[m.group(1)] = m.group(2)
    if fields.get("kernel_hash") != kernel_hash() or fields.get("workload") != workload:
        return None
    return float(fields["traffic_bytes_per_epoch"])


def algorithmic_bytes_per_epoch(n: int, dim: int, nnz: int, active: float, neg_rate: int) -> float:
    """Bytes one epoch must move at least (pull form, fp32 / int32): eps of every
    kept edge, col of each sampled edge, row_ptr + read y_i + write y_i' per
    vertex, and one dim-vector gather per positive sample and per negative."""
    return 4.0 * nnz + 4.0 * active + (4.0 + 8.0 * dim) * n + 4.0 * dim * active + 4.0 * dim * neg_rate * active


def hierarchical_roofline(n: int, dim: int, nnz: int, active: float, neg_rate: int, epoch_us: float) -> dict:
    """T* = the slowest tier's time for one epoch's algorithmic work at that tier's peak, and T* over the
    measured epoch: the edge and row streams (the algorithmic bytes without the vertex gathers) against
    HBM, and every vertex gather (one per sampled edge and per drawn negative, a random line request
    each) against the L2's request rate."""
    stream = 4.0 * nnz + 4.0 * active + (4.0 + 8.0 * dim) * n
    gathers = active * (1.0 + neg_rate)
    t_hbm = stream / (HBM_PEAK_GBPS * 1e3)                # bytes / (bytes per us)
    t_l2 = gathers / (L2_REQUEST_PEAK_G_PER_S * 1e3)       # requests / (requests per us)
    t_star = max(t_hbm, t_l2)
    return {
        "t_star_us": t_star,
        "t_measured_us": epoch_us,
        "frac": t_star / epoch_us,
        "bound": "l2-requests" if t_l2 >= t_hbm else "hbm",
        "tiers": {
            "hbm": {"bytes": stream, "peak_GBps": HBM_PEAK_GBPS, "t_us": t_hbm},
            "l2": {"requests": gathers, "peak_G_per_s": L2_REQUEST_PEAK_G_PER_S, "t_us": t_l2},
        },
    }


def build_input(w, torch, U):
    from paper_2008_00325_amd import synth

    t0 = time.time()
    step = 2_000_000
    mark = [step]

    def progress(rows):
        if rows >= mark[0]:
            log(f"kNN lists: {rows} of {w.n} rows ({time.time() - t0:.0f} s)")
            mark[0] = rows + step

    ids, dist = synth.workload_knn(w, progress if w.n > 4 * step else None)
    log(f"generated kNN lists {ids.shape} in {time.time() - t0:.1f}s")
    n, k = w.n, w.k
    di = torch.from_numpy(ids).cuda()
    dd = torch.from_numpy(dist).cuda()
    rows = torch.empty(2 * n * k, dtype=torch.int32, device="cuda")
    cols = torch.empty_like(rows)
    vals = torch.empty(2 * n * k, dtype=torch.float32, device="cuda")
    U.umap_fuzzy_graph_device(n, k, di, dd, rows, cols, vals)
    # the device fuzzy graph (smooth kNN, membership, union), timed on a second call
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    U.umap_fuzzy_graph_device(n, k, di, dd, rows, cols, vals)
    e1.record()
    torch.cuda.synchronize()
    build_input.fuzzy_graph_ms = e0.elapsed_time(e1)
    del di, dd
    a, b = U.umap_fit_ab(w.spread, w.min_dist)
    return ids, dist, rows, cols, vals, a, b


def gpu_steps(w, torch, U, coo, a, b, steps: int, warmup: int):
    rows, cols, vals = coo
    nnz = rows.numel()
    out = torch.empty((w.n, w.dim), dtype=torch.float32, device="cuda")

    def one_step(seed):
        with U.umap_layout_create_device(w.n, w.dim, rows, cols, vals, nnz, a, b, w.n_epochs, w.neg_rate) as h:
            U.umap_layout_run(h, seed)
            U.umap_layout_get_device(h, out)
            st = U.umap_layout_stats(h)
        return st

    for s in range(warmup):
        st = one_step(1000 + s)
        log(f"warmup step {s}: epochs {st['epochs_ms']:.2f} ms, ingest {st['prep_ms']:.2f} ms")
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for s in range(steps):
        stats.append(one_step(s))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for s, st in enumerate(stats):
        log(f"step {s}: epochs {st['epochs_ms']:.2f} ms, init {st['init_ms']:.3f} ms, ingest {st['prep_ms']:.2f} ms, "
            f"{st['edge_updates']} edge updates")
    ok = bool(torch.isfinite(out).all().item())
    gpu_steps.layout = out
    return stats, wall, ok


def async_mode(w, torch, U, coo, a, b, reps: int = 3) -> dict:
    """The asynchronous (Hogwild) mode on the same input, outside the timed
    steps, with each of its two kernels: median device time of the epochs over
    `reps` runs."""
    rows, cols, vals = coo
    out = {}
    with U.umap_layout_create_device(w.n, w.dim, rows, cols, vals, rows.numel(), a, b, w.n_epochs, w.neg_rate) as h:
        U.umap_layout_set_mode(h, U.UMAP_MODE_ASYNC)
        for kernel, name in ((0, "range_ordered"), (1, "per_edge")):
            U.umap_layout_set_kernel(h, kernel)
            runs = []
            for s in range(reps):
                U.umap_layout_run(h, 2000 + s)
                runs.append(U.umap_layout_stats(h))
            finite = bool(np.isfinite(U.umap_layout_get(h)).all())
            ms = float(np.median([r["epochs_ms"] for r in runs]))
            log(f"asynchronous mode, {name} kernel: epochs {ms:.2f} ms (median of {reps})")
            out[name] = {"epochs_ms": ms, "edge_updates_per_s": runs[-1]["edge_updates"] / (ms * 1e-3),
                         "finite": finite}
    out["note"] = ("asynchronous in-place (Hogwild) updates; range_ordered = the synchronous mode's launches "
                   "adding their sums in place (the default), per_edge = one lane per sampled edge applying its "
                   "attraction and negatives in turn; not bit-repeatable, quality checked by the tests "
                   "(trustworthiness within 0.01 of the oracle's)")
    return out


def shard_measure(w, U, coo, a, b, parts: int = 8, reps: int = 3) -> dict:
    """One GPU's share of a layout sharded by contiguous row ranges of about
    equal kept edges (each GPU would read the whole snapshot and write its
    rows; an all-gather of the rows would end each epoch): the epochs of each
    range on this GPU, outside the timed steps, median device time over `reps`
    runs.  The slowest range bounds the epoch of a sharded run."""
    rows, cols, vals = coo
    with U.umap_layout_create_device(w.n, w.dim, rows, cols, vals, rows.numel(), a, b, w.n_epochs, w.neg_rate) as h:
        row_ptr, _, _ = U.umap_layout_get_graph(h)
        nnz = int(row_ptr[-1])
        bounds = np.searchsorted(row_ptr, (np.arange(parts + 1, dtype=np.int64) * nnz) // parts, side="left")
        bounds[0], bounds[-1] = 0, w.n
        full = []
        for s in range(reps):
            U.umap_layout_run(h, 4000 + s)
            full.append(U.umap_layout_stats(h)["epochs_ms"])
        shards = []
        for p in range(parts):
            r0, r1 = int(bounds[p]), int(bounds[p + 1])
            U.umap_layout_set_rows(h, r0, r1)
            runs = []
            for s in range(reps):
                U.umap_layout_run(h, 4000 + s)
                runs.append(U.umap_layout_stats(h))
            ms = float(np.median([x["epochs_ms"] for x in runs]))
            shards.append({"rows": [r0, r1], "edges": int(row_ptr[r1] - row_ptr[r0]), "epochs_ms": ms,
                           "waves": runs[-1]["n_waves"],
                           "edge_updates_per_s": runs[-1]["edge_updates"] / (ms * 1e-3)})
        U.umap_layout_set_rows(h, 0, w.n)
    full_ms = float(np.median(full))
    slowest = max(x["epochs_ms"] for x in shards)
    log(f"row ranges: {parts} shares, slowest {slowest:.2f} ms vs {full_ms:.2f} ms for all rows")
    return {
        "parts": parts,
        "all_rows_epochs_ms": full_ms,
        "slowest_share_epochs_ms": slowest,
        "share_efficiency": full_ms / (parts * slowest),
        "shares": shards,
        "note": "each share's epochs run alone on this GPU, gathering from the full snapshot (rows outside the "
                "range held fixed); no all-gather and no second GPU are involved; share_efficiency = all-rows "
                "time / (parts x slowest share)",
    }


def transform_measure(w, U, table: np.ndarray, a: float, b: float, n_new: int = 100_000, n_epochs: int = 100,
                      reps: int = 3) -> dict:
    """A transform of n_new new points against the fit's layout (frozen),
    outside the timed steps: median device time of its epochs."""
    from paper_2008_00325_amd import synth

    r, c, v = synth.transform_graph(n_new, table.shape[0], w.k)
    with U.umap_transform_create(n_new, table, r, c, v, a, b, n_epochs, w.neg_rate) as h:
        runs = []
        for s in range(reps):
            U.umap_layout_run(h, 3000 + s)
            runs.append(U.umap_layout_stats(h))
        finite = bool(np.isfinite(U.umap_layout_get(h)).all())
    ms = float(np.median([x["epochs_ms"] for x in runs]))
    log(f"transform: {n_new} points, {n_epochs} epochs in {ms:.2f} ms")
    return {
        "n_new": n_new, "n_table": int(table.shape[0]), "k": w.k, "n_epochs": n_epochs,
        "epochs_ms": ms,
        "edge_updates_per_s": runs[-1]["edge_updates"] / (ms * 1e-3),
        "table_ranges": runs[-1]["table_ranges"],
        "finite": finite,
        "note": "new points with k edges each into a +-64 window of the fit's layout, weights uniform on "
                "[0.05, 1); only the new points move",
    }


def trustworthiness_measure(torch, U, n: int = 70_000, d: int = 784, k: int = 15, reps: int = 2) -> dict:
    """The GPU trustworthiness on the 70,000 x 784 image-like points and a
    random 2-D embedding: its dominant work is the n x n input distances as
    fp32 MFMA tiles (2 n^2 d flops)."""
    from paper_2008_00325_amd import synth

    X, _ = synth.image_like(n, d)
    Xg = torch.from_numpy(X).cuda()
    Yg = torch.from_numpy(synth.embedding_state(n, 2, 1)).cuda()
    U.umap_trustworthiness(Xg, Yg, k)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        U.umap_trustworthiness(Xg, Yg, k)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / reps * 1e3
    flops = 2.0 * n * n * d
    tflops = flops / (ms * 1e-3) / 1e12
    log(f"trustworthiness: n {n} x {d}, k {k}: {ms:.1f} ms, {tflops:.1f} TFLOP/s")
    return {
        "n": n, "d": d, "k": k, "ms": ms,
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / FP32_MFMA_PEAK_TFLOPS,
                     "note": "2 n^2 d flops of the input distances over the whole call (embedding kNN, "
                             "thresholds and rank counting included), host-timed around the blocking call"},
    }


def non_knn_at_3m(torch, U, a: float, b: float) -> dict:
    """Everything after the kNN search at the scale of the paper's largest
    single-GPU run (3M points, k = 15): the fuzzy graph, the ingest, the
    initialisation and 200 epochs in 2-D, on a synthetic window kNN graph (90
    clusters of ~33k vertices, the window1m recipe at 3M vertices).  Device
    times from HIP events and the library's stats."""
    from paper_2008_00325_amd import synth

    n, k, n_epochs, neg_rate = 3_000_000, 15, 200, 5
    ids, dist = synth.window_knn(n, k, synth.cluster_bounds(n, 90), seed=7)
    di = torch.from_numpy(ids).cuda()
    dd = torch.from_numpy(dist).cuda()
    del ids, dist
    rows = torch.empty(2 * n * k, dtype=torch.int32, device="cuda")
    cols = torch.empty_like(rows)
    vals = torch.empty(2 * n * k, dtype=torch.float32, device="cuda")
    U.umap_fuzzy_graph_device(n, k, di, dd, rows, cols, vals)   # warm-up
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    U.umap_fuzzy_graph_device(n, k, di, dd, rows, cols, vals)
    e1.record()
    torch.cuda.synchronize()
    graph_ms = e0.elapsed_time(e1)
    del di, dd
    with U.umap_layout_create_device(n, 2, rows, cols, vals, rows.numel(), a, b, n_epochs, neg_rate) as h:
        U.umap_layout_run(h, 5)
        st = U.umap_layout_stats(h)
    total_ms = graph_ms + st["prep_ms"] + st["init_ms"] + st["epochs_ms"]
    log(f"3M vertices: fuzzy graph {graph_ms:.1f} ms, ingest {st['prep_ms']:.1f} ms, init {st['init_ms']:.2f} ms, "
        f"200 epochs {st['epochs_ms']:.1f} ms: {total_ms / 1e3:.3f} s (the paper: 9.3 s of non-kNN work at 3M)")
    return {"n": n, "k": k, "n_epochs": n_epochs, "fuzzy_graph_ms": graph_ms, "ingest_ms": st["prep_ms"],
            "init_ms": st["init_ms"], "epochs_ms": st["epochs_ms"], "total_s": total_ms / 1e3,
            "nnz_kept": st["nnz_kept"], "table_ranges": st["table_ranges"],
            "paper_gv100_non_knn_s": 9.3,
            "note": "the paper's figure is all non-kNN work of its 3M-point GoogleNews run on an NVIDIA GV100 "
                    "(epochs and dimensions unstated): context on other hardware and data, not a target"}


# The paper's trustworthiness times (Table 4: isotropic blobs, 1024 features,
# k = 15; seconds on one NVIDIA GV100), quoted as context beside ours.
PAPER_TABLE4_GPU_S = {2000: 0.13, 5000: 0.18, 10000: 0.24, 20000: 0.54, 50000: 2.07, 100000: 5.74}


def trustworthiness_sizes(torch, U, sizes=(2000, 5000, 10000, 20000, 50000, 100000), d: int = 1024,
                          k: int = 15) -> dict:
    """The GPU trustworthiness at the shapes of the paper's timing table:
    isotropic blobs (5 centres, std 1) with 1024 features and a random 2-D
    embedding, host-timed around each blocking call (the best of 3 after one
    warm-up)."""
    from paper_2008_00325_amd import synth

    rows = []
    for n in sizes:
        X, _ = synth.blobs(n, d, 5, seed=n)
        Xg = torch.from_numpy(X).cuda()
        Yg = torch.from_numpy(synth.embedding_state(n, 2, 1)).cuda()
        U.umap_trustworthiness(Xg, Yg, k)
        best = float("inf")
        for _ in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            U.umap_trustworthiness(Xg, Yg, k)
            torch.cuda.synchronize()
            best = min(best, time.perf_counter() - t0)
        rows.append({"n": n, "s": best, "tflops": 2.0 * n * n * d / best / 1e12,
                     "paper_gv100_s": PAPER_TABLE4_GPU_S.get(n)})
        log(f"trustworthiness {n} x {d}: {best * 1e3:.1f} ms (the paper's GV100: {PAPER_TABLE4_GPU_S.get(n)} s)")
        del Xg, Yg
    return {"d": d, "k": k, "rows": rows,
            "note": "the paper's column is its own implementation on an NVIDIA GV100 (context, other hardware)"}


def copy_probe(torch, U, mb: int = 1024, reps: int = 5) -> float:
    """HBM copy bandwidth of the library's plain 16-byte copy kernel (GB/s,
    read + write bytes), on the current stream."""
    nbytes = mb * 1024 * 1024
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream()
    U.umap_probe_copy(src, dst, nbytes, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        U.umap_probe_copy(src, dst, nbytes, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return 2.0 * nbytes / (ms * 1e-3) / 1e9


def gather_probe(torch, U, table_bytes: int, reps: int = 3) -> float:
    """Random 8-byte gathers per second from a table of `table_bytes` (the
    library's gather probe: the repulsions' access pattern without their
    arithmetic), on the current stream."""
    entries = table_bytes // 8
    table = torch.ones(entries * 2, dtype=torch.float32, device="cuda")
    threads, iters = 8192 * 256, 8
    out = torch.empty(threads, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    U.umap_probe_gather(table, entries, threads, iters, out, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        U.umap_probe_gather(table, entries, threads, iters, out, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return threads * iters * 16 / (ms * 1e-3)


def host_cpu() -> dict:
    """The host the oracle ran on: CPU model, sockets and cores (lscpu), the
    processor count and the cores this process may use."""
    info = {"nproc": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0))}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        fields = dict(line.split(":", 1) for line in out.splitlines() if ":" in line)
        for key, name in (("Model name", "model"), ("Socket(s)", "sockets"), ("Core(s) per socket", "cores_per_socket"),
                          ("Thread(s) per core", "threads_per_core"), ("CPU max MHz", "max_mhz")):
            if key in fields:
                info[name] = fields[key].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    if "model" not in info:
        try:
            with open("/proc/cpuinfo") as f:
                for line in f:
                    if line.startswith("model name"):
                        info["model"] = line.split(":", 1)[1].strip()
                        break
        except OSError:
            pass
    return info


def cpu_baseline(w, ids, dist, budget_s: float = 12.0):
    """The C oracle (fp64 push-form Jacobi epochs) timed on the host cores, on
    a sample of epochs spread over the run, from the random initial layout."""
    import oracle as O

    t0 = time.time()
    r, c, v = O.fuzzy_graph(ids, dist)
    g = O.prep(w.n, r, c, v, w.n_epochs)
    a, b = O.fit_ab(w.spread, w.min_dist)
    E = O.init_layout(w.n, w.dim, 0).astype(np.float64)
    log(f"oracle graph ready in {time.time() - t0:.1f}s ({g.nnz} edges); timing epochs")
    # epochs spread over the run (bisection order) until about budget_s of CPU time
    sample, seen = [], set()
    step = w.n_epochs
    while step >= 1 and len(sample) < w.n_epochs:
        for ep in range(0, w.n_epochs, step):
            if ep not in seen:
                seen.add(ep)
                sample.append(ep)
        step //= 2
    done, updates, spent = [], 0, 0.0
    for ep in sample:
        t1 = time.perf_counter()
        _, act = O.epoch(g, E, ep, a, b, w.n_epochs, w.neg_rate, 0)
        spent += time.perf_counter() - t1
        updates += act * (1 + w.neg_rate)
        done.append(ep)
        if spent > budget_s:
            break
    cores = O.num_threads()
    # one thread on the middle epoch of the run
    mid = w.n_epochs // 2
    O.set_num_threads(1)
    try:
        t1 = time.perf_counter()
        _, act1 = O.epoch(g, E, mid, a, b, w.n_epochs, w.neg_rate, 0)
        one = act1 * (1 + w.neg_rate) / (time.perf_counter() - t1)
    finally:
        O.set_num_threads(cores)
    log(f"oracle: {updates / spent:.3g} edge-updates/s on {cores} threads, {one:.3g} on one")
    return {
        "value": updates / spent,
        "unit": "edge-updates/s",
        "cores": cores,
        "kind": "oracle",
        "host": host_cpu(),
        "sample": f"{len(done)} of the {w.n_epochs} epochs of the {w.name} layout (spread over the run: "
                  f"{done[:6]}...), each from the random initial layout; fp64 push form, "
                  f"{updates} edge updates in {spent:.2f} s",
        "single_thread_value": one,
        "single_thread_sample": f"epoch {mid} from the random initial layout on one thread",
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="window1m")
    ap.add_argument("--n-components", type=int, default=0,
                    help="embedding dimension in place of the workload's own (same graph)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extras", action="store_true",
                    help="also measure the asynchronous mode, one GPU's row share, the transform and the GPU "
                         "trustworthiness (the rows beyond the layout epochs)")
    ap.add_argument("--context", action="store_true",
                    help="also measure the context figures at the shapes of the paper's own experiments (all "
                         "non-kNN work at 3M points; trustworthiness at the shapes of its timing table)")
    ap.add_argument("--no-extras", action="store_true",
                    help="the default (kept so that recorded profiling commands stay valid)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the layout is measured on a single MI355X); got --gpus {args.gpus}",
              file=sys.stderr)
        return 2

    import torch

    from paper_2008_00325_amd import synth
    from paper_2008_00325_amd import umap_layout as U

    U.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    w = synth.WORKLOADS[args.workload]
    if args.n_components:
        w = dataclasses.replace(w, dim=args.n_components)
    ids, dist, rows, cols, vals, a, b = build_input(w, torch, U)
    stats, wall, finite = gpu_steps(w, torch, U, (rows, cols, vals), a, b, args.steps, args.warmup)
    if not finite:
        log("non-finite layout")
        return 1
    updates = sum(s["edge_updates"] for s in stats)
    st = stats[-1]
    epochs_ms = float(np.median([s["epochs_ms"] for s in stats]))
    prep_ms = float(np.median([s["prep_ms"] for s in stats]))
    init_ms = float(np.median([s["init_ms"] for s in stats]))
    n_epochs = st["n_epochs"]
    avg_active = st["active_edges"] / n_epochs
    bytes_epoch = algorithmic_bytes_per_epoch(w.n, w.dim, st["nnz_kept"], avg_active, w.neg_rate)
    launch_ms = epochs_ms / n_epochs
    achieved = bytes_epoch / (launch_ms * 1e-3) / 1e9
    traffic = profiled_traffic(w.name)
    extras = {}
    if args.extras and not args.no_extras:
        extras["async_mode"] = async_mode(w, torch, U, (rows, cols, vals), a, b)
        extras["row_shares"] = shard_measure(w, U, (rows, cols, vals), a, b)
        extras["transform"] = transform_measure(w, U, gpu_steps.layout.cpu().numpy(), a, b)
        extras["trustworthiness"] = trustworthiness_measure(torch, U)
    if args.context and not args.no_extras:
        extras["non_knn_at_3m"] = non_knn_at_3m(torch, U, a, b)
        extras["trustworthiness_paper_table4_shapes"] = trustworthiness_sizes(torch, U)
    copy_gbps = copy_probe(torch, U)
    range_bytes = (w.n * w.dim * 4) // st["table_ranges"]
    table_pow2 = 1 << max(3, (range_bytes - 1).bit_length())
    gather_range = gather_probe(torch, U, table_pow2)
    gather_full = gather_probe(torch, U, 1 << max(3, (w.n * w.dim * 4 - 1).bit_length()))
    # gathers per epoch: a positive sample and neg_rate drawn negatives per sampled edge
    gathers_per_s = st["edge_updates"] / (epochs_ms * 1e-3)
    props = torch.cuda.get_device_properties(0)
    gpu_name = f"{props.name} ({getattr(props, 'gcnArchName', '?')}, {props.multi_processor_count} CUs)"

    result = {
        "metric": "SGD edge-updates/sec (pos+neg) and 200-epoch layout wall time at 1M points",
        "value": updates / wall,
        "unit": "edge-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "n": w.n, "k": w.k, "n_components": w.dim, "n_epochs": w.n_epochs,
            "neg_rate": w.neg_rate, "min_dist": w.min_dist, "spread": w.spread, "a": a, "b": b,
            "nnz_input": st["nnz_input"], "nnz_kept": st["nnz_kept"], "max_degree": st["max_degree"],
            "step": "device ingest + init + all epochs + device copy-out",
        },
        "layout_wall_s": epochs_ms * 1e-3,
        "layout_epochs_updates_per_s": st["edge_updates"] / (epochs_ms * 1e-3),
        "ingest_ms": prep_ms,
        "init_ms": init_ms,
        "edge_updates_per_step": st["edge_updates"],
        "roofline": {
            "bound": "hbm",
            "kernel": f"epoch = k_epoch_draw + {st['table_ranges']} x k_epoch_repulse",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": bytes_epoch,
            "avg_launch_ms": launch_ms,
        },
        "gather_roofline": {
            "bound": "l2-gather",
            "achieved": gathers_per_s / 1e9,
            "peak": gather_range / 1e9,
            "unit": "G gathers/s",
            "frac": gathers_per_s / gather_range,
            "note": f"8-byte vertex gathers of the epoch (one per positive sample and drawn negative) over the "
                    f"epochs time, against the library's gather probe on a {table_pow2 >> 20} MB table (one "
                    f"vertex-table range, the slice one repulsion launch gathers from); the probe on the whole "
                    f"{w.n * w.dim * 4 / 1e6:.0f} MB table reaches {gather_full / 1e9:.0f} G/s",
        },
        "hierarchical_roofline": {
            **hierarchical_roofline(w.n, w.dim, st["nnz_kept"], avg_active, w.neg_rate, launch_ms * 1e3),
            "note": f"L2 request peak from the chip's structure (8 XCDs x 16 channels x 2.4 GHz); the "
                    f"library's gather probe on a {table_pow2 >> 20} MB table reaches "
                    f"{gather_range / 1e9 / L2_REQUEST_PEAK_G_PER_S:.2f} of it",
        },
        **extras,
        "fuzzy_graph_ms": build_input.fuzzy_graph_ms,
        "hbm_copy_probe_GBps": copy_gbps,
        "gpu": gpu_name,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, ids, dist)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
