"""Host logic of the benchmark (no GPU): the busy time of overlapping transfer intervals, and the
lookup of counter-measured traffic, which must return nothing once a kernel's source differs
from the one the counters were taken on."""
import os
import shutil

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
    rec = bench.traffic_record("dsa_mla_32req_8L_ctx32K_k2048_B4096", "fetch")
    assert rec is not None and rec["fetch_bytes"] > 0 and rec["write_bytes"] > 0
    assert bench.traffic_record("no_such_workload", "fetch") is None
    # a copy of the tree where one source of the kernel differs by a byte: no record applies
    for d in ("profiles", "paper_2608_07009_amd/csrc"):
        shutil.copytree(os.path.join(bench.ROOT, d), tmp_path / d)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_record("dsa_mla_32req_8L_ctx32K_k2048_B4096", "fetch") == \
        dict(rec, profile=rec["profile"])
    src = tmp_path / "paper_2608_07009_amd/csrc/fetch_device.h"
    src.write_bytes(src.read_bytes() + b"\n")
    assert bench.traffic_record("dsa_mla_32req_8L_ctx32K_k2048_B4096", "fetch") is None
