"""Host logic of the benchmark (no GPU): the busy time of overlapping transfer intervals, the
lookup of counter-measured traffic, which must return nothing once a kernel's source differs
from the one the counters were taken on, the threaded CPU baseline, and the default run's child
process per workload."""
import os

import numpy as np

import bench


def brute_union(intervals, step=1e-3):
    """Length of the union by sampling a fine grid (intervals on multiples of `step`)."""
    if not intervals:
        return 0.0
    lo = min(a for a, _ in intervals)
    hi = max(b for _, b in intervals)
    n = int(round((hi - lo) / step))
    covered = np.zeros(n, dtype=bool)
    for a, b in intervals:
        covered[int(round((a - lo) / step)):int(round((b - lo) / step))] = True
    return covered.sum() * step


def test_union_length_matches_brute_force():
    rng = np.random.default_rng(5)
    assert bench.union_length([]) == 0.0
    assert bench.union_length([(0.0, 1.0), (1.0, 2.0)]) == 2.0      # touching
    assert bench.union_length([(0.0, 3.0), (1.0, 2.0)]) == 3.0      # nested
    assert bench.union_length([(2.0, 3.0), (0.0, 1.0)]) == 2.0      # disjoint, unsorted
    for _ in range(200):
        iv = []
        for _ in range(int(rng.integers(1, 12))):
            a = int(rng.integers(0, 400))
            iv.append((a * 1e-3, (a + int(rng.integers(1, 80))) * 1e-3))
        assert abs(bench.union_length(iv) - brute_union(iv)) < 1e-9


def test_traffic_record_follows_the_kernel_sources(tmp_path, monkeypatch):
    """A synthetic record over two synthetic source files: it applies while their bytes hash to
    the recorded sha256 and stops applying as soon as one of them changes."""
    import hashlib
    (tmp_path / "profiles").mkdir()
    (tmp_path / "src").mkdir()
    a, b = tmp_path / "src" / "k.hip", tmp_path / "src" / "k.h"
    a.write_bytes(b"__global__ void k() {}\n")
    b.write_bytes(b"#pragma once\n")
    sha = hashlib.sha256(a.read_bytes() + b.read_bytes()).hexdigest()
    (tmp_path / "profiles" / "k.md").write_text(
        "# synthetic\n\ntraffic-record workload=w1 kernel=fetch source=src/k.hip,src/k.h "
        f"sha256={sha} fetch_bytes=1200 write_bytes=1100\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = bench.traffic_record("w1", "fetch")
    assert rec == {"fetch_bytes": 1200, "write_bytes": 1100, "profile": "profiles/k.md"}
    assert bench.traffic_record("w2", "fetch") is None
    assert bench.traffic_record("w1", "sparse_decode") is None
    b.write_bytes(b.read_bytes() + b"\n")  # one byte more in one source: the record is stale
    assert bench.traffic_record("w1", "fetch") is None
    b.unlink()  # a missing source: no record either
    assert bench.traffic_record("w1", "fetch") is None


def test_cpu_baseline_runs_every_unit_on_threads():
    """The CPU baseline resolves every (anchor layer, unit) stream on a pool of threads over
    disjoint units and times float64 attention apart; its figures are positive and its resolve
    covers whole steps."""
    import workload as W
    w = W.workload(1, num_requests=3, num_layers=2)
    host = np.empty((w.num_layers, w.units, w.L, w.record_bytes), dtype=np.uint8)
    for l in range(w.num_layers):
        W.fill_kv(host[l].ctypes.data, w, l, 0, w.units)
    r = bench.cpu_baseline(w, lambda layer, unit: host[layer, unit], budget_s=1.0)
    assert r["kind"] == "oracle" and r["unit"] == "selections/s" and r["value"] > 0
    assert 1 <= r["cores"] <= w.units * w.num_layers
    assert 1 <= r["resolve_steps_done"] <= r["resolve_steps_in_workload"] == w.steps
    assert r["attention_us_per_unit"] > 0 and r["cpu_model"]


def test_default_run_tries_every_workload_in_a_child(tmp_path):
    """Without --config the benchmark starts one child process per workload and never touches
    the GPU itself; here (no GPU) every child reports that, and the parent says which failed."""
    import json
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--steps", "4",
                        "--warmup", "2", "--no-sweep"], capture_output=True, text=True,
                       timeout=600, cwd=str(tmp_path))
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert r.returncode == 1 and "error" in line
    assert sorted(line["configs"]) == ["1", "2", "3", "4", "5"]
    assert all("no GPU" in v["error"] for v in line["configs"].values())


def test_compact_keeps_the_per_workload_figures():
    d = {"value": 1.0, "unit": "selections/s", "ms_per_step": 2.0, "miss_fetch_GBps": 40.0,
         "roofline": {"frac": 0.7}, "extra": 1,
         "config": {"workload": "w", "layers": 56, "layers_in_workload": 61, "requests": 1},
         "kernels": {"fetch": {"avg_us": 27.123, "launches": 3}}}
    c = bench.compact(d)
    assert c["layers"] == 56 and c["layers_in_workload"] == 61 and "extra" not in c
    assert c["roofline"] == {"frac": 0.7} and c["kernels_avg_us"] == {"fetch": 27.12}
