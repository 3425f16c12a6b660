"""Host logic of bench.py (no GPU): the single-GPU contract, the algorithmic
bytes of an epoch, the tiered roofline, and the rule that ties a profile's traffic figure to the
kernel sources it was taken on."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_algorithmic_bytes_by_hand():
    # 10 vertices in 2-D, 40 kept edges, 12 sampled, 5 negatives each:
    # eps 4 x 40, col 4 x 12, row_ptr + y_i read + y_i' write (4 + 8 x 2) x 10,
    # positive gathers 8 x 12, negative gathers 8 x 5 x 12
    want = 160 + 48 + 200 + 96 + 480
    assert bench.algorithmic_bytes_per_epoch(10, 2, 40, 12, 5) == want
    # the 1M-vertex workload's figure: 26,687,328 kept edges, 7,629,883 sampled per epoch on average
    b = bench.algorithmic_bytes_per_epoch(1_000_000, 2, 26_687_328, 7_629_882.92, 5)
    assert abs(b / 1e6 - 523.5) < 0.1


def test_hierarchical_roofline_by_hand():
    # 10 vertices in 2-D, 40 kept edges, 12 sampled, 5 negatives each: streams 160 + 48 + 200 = 408 bytes,
    # 12 x 6 = 72 vertex gathers; HBM at 8 TB/s = 8e6 bytes per us, L2 at 307.2e3 requests per us
    r = bench.hierarchical_roofline(10, 2, 40, 12, 5, epoch_us=1.0)
    assert abs(r["tiers"]["hbm"]["t_us"] - 408 / 8e6) < 1e-15
    assert abs(r["tiers"]["l2"]["t_us"] - 72 / 307.2e3) < 1e-15
    assert r["bound"] == "l2-requests" and abs(r["frac"] - 72 / 307.2e3) < 1e-15
    # the 1M-vertex workload: 157.3 MB of streams (19.7 us), 45.78 M gathers (149.0 us)
    r = bench.hierarchical_roofline(1_000_000, 2, 26_687_328, 7_629_882.92, 5, epoch_us=306.5)
    assert abs(r["tiers"]["hbm"]["t_us"] - 19.66) < 0.01
    assert abs(r["tiers"]["l2"]["t_us"] - 149.02) < 0.01
    assert abs(r["frac"] - 149.02 / 306.5) < 1e-4


def test_kernel_hash_ignores_comments(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int f() { return 1; }  // one\n/* block */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", ["k.hip"])
    h1 = bench.kernel_hash()
    src.write_text("int f() {\n  return 1;   // another comment\n}\n")
    assert bench.kernel_hash() == h1
    src.write_text("int f() { return 2; }\n")
    assert bench.kernel_hash() != h1


def test_profile_traffic_only_for_matching_sources(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int f() { return 1; }\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", ["k.hip"])
    prof = tmp_path / "p.md"
    prof.write_text(f"- workload: `window1m`\n- kernel_hash: `{bench.kernel_hash()}` (note)\n"
                    f"- traffic_bytes_per_epoch: `813000000`\n")
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", str(prof))
    assert bench.profiled_traffic("window1m") == 813000000.0
    assert bench.profiled_traffic("window5m") is None
    src.write_text("int f() { return 3; }\n")
    assert bench.profiled_traffic("window1m") is None


def test_committed_profile_matches_committed_kernels():
    """The profile summary in the repository was taken on the epoch kernels in
    the repository, so the bench line carries its measured traffic."""
    assert bench.profiled_traffic("window1m") is not None
