"""Cache-size study on the synthetic selection streams (CPU; Section 4.3's replacement-policy
comparison, run on the stand-in streams since the paper's trace is not available).

LRU is the oracle's canonical policy. Pins for the comparison models: the offline optimum
(BELADY) never misses more than any online policy; B = k staging misses exactly
|S_t \\ S_{t-1}| and so does LRU at B = k; with B >= L nothing is ever evicted, so every policy
misses only first touches. Run with -s to print the miss-rate table for the 32K-context DSA/MLA streams."""
import numpy as np
import pytest

import oracle
import workload as W
from policy_models import misses

POLICIES = ("LRU", "FIFO", "RANDOM", "BELADY")


def lru_misses(stream, B, L):
    c = oracle.OracleCache(1, L, B, stream.shape[1])
    return np.array([int(c.resolve_unit(0, s.astype(np.int32))[2][1]) for s in stream])


def policy_misses(stream, B, L, policy, seed=0):
    return lru_misses(stream, B, L) if policy == "LRU" else misses(stream, B, policy, seed)


def test_belady_is_optimal_and_closed_forms():
    rng = np.random.default_rng(11)
    for trial in range(20):
        L = int(rng.integers(16, 80))
        k = int(rng.integers(2, 10))
        B = int(rng.integers(k, 3 * k))
        steps = 25
        stream = np.stack([rng.choice(L, size=k, replace=False) for _ in range(steps)])
        got = {p: policy_misses(stream, B, L, p, seed=trial) for p in POLICIES}
        for p in ("LRU", "FIFO", "RANDOM"):
            assert got["BELADY"].sum() <= got[p].sum()
        topk = misses(stream, k, "TOPK")
        assert topk.tolist() == [len(set(stream[0]))] + [
            len(set(stream[t]) - set(stream[t - 1])) for t in range(1, steps)]
        assert lru_misses(stream, k, L).tolist() == topk.tolist()  # B = k: top-k staging
        big = {p: policy_misses(stream, L, L, p).sum() for p in POLICIES}
        assert len(set(big.values())) == 1 and big["LRU"] == len(set(stream.ravel().tolist()))


def test_miss_rates_on_dsa_streams():
    w = W.workload(2, num_requests=1, num_layers=1)
    steps = 48
    stream = W.selection_streams(w, steps=steps)[:, 0, :]
    rows = []
    for ratio in (1, 1.5, 2, 4):
        B = int(w.k * ratio)
        m = {p: policy_misses(stream, B, w.L, p, seed=1)[8:].mean() / w.k for p in POLICIES}
        rows.append((ratio, m))
        assert m["BELADY"] <= min(m["LRU"], m["FIFO"], m["RANDOM"]) + 1e-12
    print("\nmiss rate per step after warm-up (32K-context DSA/MLA streams, k = 2048)")
    print("B/k  " + "  ".join(f"{p:>7s}" for p in POLICIES))
    for ratio, m in rows:
        print(f"{ratio:<4} " + "  ".join(f"{m[p]:7.4f}" for p in POLICIES))
    # more cache never hurts LRU on these streams (stack property of LRU)
    lru = [m["LRU"] for _, m in rows]
    assert all(a >= b for a, b in zip(lru, lru[1:]))
