"""Set-based cache replacement models for the cache-size study (test infrastructure).

The canonical LRU is the oracle's; these are the comparison policies. Each model serves one
unit's selection stream: at every step the whole selected set must be
resident in B slots; selected positions that are not resident are misses and evict
non-selected residents chosen by the policy. They count misses only (no slot numbering).
  * FIFO    - least recently admitted first;
  * RANDOM  - uniformly random non-selected resident (seeded);
  * BELADY  - the non-selected resident whose next selection is farthest in the future
              (offline optimum for this access pattern);
  * TOPK    - B = k staging: the cache holds exactly the current selection.
"""
from __future__ import annotations

import numpy as np


def misses(stream: np.ndarray, B: int, policy: str, seed: int = 0) -> np.ndarray:
    """stream: int [steps][k] positions (>= 0). Returns misses per step."""
    steps = stream.shape[0]
    sets = [set(int(p) for p in s if p >= 0) for s in stream]
    rng = np.random.default_rng(seed)
    if policy == "TOPK":
        out, prev = [], set()
        for S in sets:
            out.append(len(S - prev))
            prev = S
        return np.array(out)
    # next use of each position after step t (BELADY)
    next_use = {}
    nxt = []
    for t in range(steps - 1, -1, -1):
        nxt.append({p: next_use.get(p, steps + 1) for p in sets[t]})
        for p in sets[t]:
            next_use[p] = t
    nxt.reverse()  # nxt[t][p] = next step after t that selects p
    resident = {}  # position -> key (admission step for FIFO, next use for BELADY)
    out = []
    for t, S in enumerate(sets):
        miss = [p for p in S if p not in resident]
        free = B - len(resident)
        need = max(0, len(miss) - free)
        if need:
            cand = [p for p in resident if p not in S]
            if policy == "RANDOM":
                victims = rng.choice(len(cand), size=need, replace=False)
                victims = [cand[i] for i in victims]
            elif policy == "BELADY":
                victims = sorted(cand, key=lambda p: -resident[p])[:need]
            else:  # FIFO: earliest admission first
                victims = sorted(cand, key=lambda p: resident[p])[:need]
            for p in victims:
                del resident[p]
        for p in S:
            if policy == "FIFO":
                resident.setdefault(p, t)
            elif policy == "BELADY":
                resident[p] = nxt[t][p]
            else:
                resident.setdefault(p, 0)
        out.append(len(miss))
    return np.array(out)
