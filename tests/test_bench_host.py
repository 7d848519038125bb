"""Host logic of the benchmark (no GPU): the busy time of overlapping transfer intervals, and the
lookup of counter-measured traffic, which must return nothing once a kernel's source differs
from the one the counters were taken on."""
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
