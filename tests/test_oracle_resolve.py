"""Pins for the oracle's resolve step (CPU only).

The oracle (oracle/hisparse_oracle.c) is checked against things other than itself:
  * a worked example derived by hand from the replacement policy (tests/golden);
  * closed forms the paper's policy fixes: cold start, top-k-only staging B = k (Section 4.3,
    the "Swap-vanilla" configuration: the cache then holds exactly the current selection), and
    B >= L (nothing is ever evicted);
  * an independent list-based LRU model (move-to-front recency list instead of timestamps);
  * invariants of Section 3.1/3.2: every selected record is resident after resolve, the page
    table and slot map are mutual inverses, occupancy <= B, hits + misses = |S|, no slot hit
    this step is a victim.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lru_worked_example.json")


class ListLRU:
    """Independent model of the policy: an explicit recency list of slots (least recent first),
    initially the empty slots in slot order. Per step, victims are the least recent slots not
    hit; the new list is [untouched, in old order] + [victims by slot] + [hit slots by slot]."""

    def __init__(self, B):
        self.B = B
        self.where = {}
        self.content = [None] * B
        self.recency = list(range(B))

    def step(self, sel):
        S = [int(p) for p in sel if p >= 0]
        hit_slots = sorted(self.where[p] for p in S if p in self.where)
        misses = sorted(p for p in S if p not in self.where)
        hs = set(hit_slots)
        victims = [s for s in self.recency if s not in hs][:len(misses)]
        for p, v in zip(misses, victims):
            if self.content[v] is not None:
                del self.where[self.content[v]]
            self.content[v] = p
            self.where[p] = v
        touched = hs | set(victims)
        self.recency = [s for s in self.recency if s not in touched] + sorted(victims) + hit_slots
        slots = [self.where[int(p)] if p >= 0 else -1 for p in sel]
        return slots, (len(hit_slots), len(misses)), list(zip(misses, victims))


def test_worked_example():
    g = json.load(open(GOLDEN))
    c = oracle.OracleCache(1, g["L"], g["B"], g["k"])
    for st in g["steps"]:
        rc, slots, counts, pp, ps = c.resolve_unit(0, np.array(st["sel"]))
        assert rc == oracle.OK
        assert slots.tolist() == st["slots"]
        assert counts.tolist() == st["counts"]
        assert [list(x) for x in zip(pp.tolist(), ps.tolist())] == st["plan"]
        assert c.slot_pos[0].tolist() == st["slot_pos"]
        assert c.slot_ts[0].tolist() == st["slot_ts"]


def test_hits_outrank_same_step_misses():
    # Section 3.2: a record selected repeatedly outranks a first-time selection.
    # B=2: step 1 fetches 0 and 1; step 2 hits 0 and fetches 2 (evicting 1); step 3 needs one
    # victim: 2 (a miss of step 2) must go before 0 (a hit of step 2).
    c = oracle.OracleCache(1, 8, 2, 2)
    c.resolve_unit(0, np.array([0, 1]))
    c.resolve_unit(0, np.array([0, 2]))
    rc, slots, counts, pp, ps = c.resolve_unit(0, np.array([5, -1]))
    assert counts.tolist() == [0, 1]
    assert 0 in c.slot_pos[0] and 2 not in c.slot_pos[0] and 5 in c.slot_pos[0]


def test_cold_start_closed_form():
    rng = np.random.default_rng(1)
    for _ in range(50):
        L, B = 200, 64
        k = int(rng.integers(1, B + 1))
        sel = rng.choice(L, size=k, replace=False).astype(np.int32)
        c = oracle.OracleCache(1, L, B, k)
        rc, slots, counts, pp, ps = c.resolve_unit(0, sel)
        order = np.argsort(sel)
        # the i-th smallest position lands in slot i
        assert (slots[order] == np.arange(k)).all()
        assert counts.tolist() == [0, k]


def _random_stream(rng, L, k, steps, overlap):
    prev = rng.choice(L, size=k, replace=False)
    out = [prev]
    for _ in range(steps - 1):
        keep = rng.choice(prev, size=int(overlap * k), replace=False)
        pool = np.setdiff1d(np.arange(L), keep)
        new = rng.choice(pool, size=k - len(keep), replace=False)
        cur = rng.permutation(np.concatenate([keep, new]))
        out.append(cur)
        prev = cur
    return [s.astype(np.int32) for s in out]


def test_topk_only_staging_closed_form():
    # B = k: the cache holds exactly S_t after step t, so misses_t = |S_t \ S_{t-1}|.
    rng = np.random.default_rng(2)
    L, k = 300, 40
    stream = _random_stream(rng, L, k, 30, 0.6)
    c = oracle.OracleCache(1, L, k, k)
    prev = set()
    for s in stream:
        rc, slots, counts, pp, ps = c.resolve_unit(0, s)
        assert counts[1] == len(set(s.tolist()) - prev)
        assert set(c.slot_pos[0].tolist()) == set(s.tolist())
        prev = set(s.tolist())


def test_no_eviction_when_cache_covers_context():
    # B >= L: misses_t = |S_t \ union of earlier S|; every fetch lands in a fresh slot.
    rng = np.random.default_rng(3)
    L, k = 64, 16
    stream = _random_stream(rng, L, k, 25, 0.3)
    c = oracle.OracleCache(1, L, L, k)
    seen = set()
    used = set()
    for s in stream:
        rc, slots, counts, pp, ps = c.resolve_unit(0, s)
        assert counts[1] == len(set(s.tolist()) - seen)
        assert not (set(ps.tolist()) & used)
        used |= set(ps.tolist())
        seen |= set(s.tolist())


@pytest.mark.parametrize("seed", range(6))
def test_matches_list_lru_and_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    for trial in range(60):
        L = int(rng.integers(4, 64))
        B = int(rng.integers(1, 17))
        k = int(rng.integers(1, min(B, L) + 1))
        steps = int(rng.integers(1, 30))
        model = ListLRU(B)
        c = oracle.OracleCache(1, L, B, k)
        for t in range(steps):
            nvalid = int(rng.integers(0, k + 1))
            sel = np.full(k, -1, dtype=np.int32)
            sel[:nvalid] = rng.choice(L, size=nvalid, replace=False)
            sel = rng.permutation(sel).astype(np.int32)
            rc, slots, counts, pp, ps = c.resolve_unit(0, sel)
            e_slots, e_counts, e_plan = model.step(sel)
            assert rc == oracle.OK
            assert slots.tolist() == e_slots
            assert tuple(counts.tolist()) == e_counts
            assert list(zip(pp.tolist(), ps.tolist())) == e_plan
            # invariants
            pt, sp = c.pt[0], c.slot_pos[0]
            valid = sel[sel >= 0]
            assert counts.sum() == len(valid)
            assert (sp[slots[sel >= 0]] == valid).all()
            assert (slots[sel < 0] == -1).all()
            assert len(set(slots[sel >= 0].tolist())) == len(valid)
            res = np.nonzero(sp >= 0)[0]
            assert (pt[sp[res]] == res).all()
            assert (pt >= 0).sum() == len(res) <= B
            hit_slots = set(slots[sel >= 0].tolist()) - set(ps.tolist())
            assert not (hit_slots & set(ps.tolist()))
            assert int(c.clock[0]) == t + 1


def test_multi_unit_matches_single_unit():
    rng = np.random.default_rng(7)
    U, L, B, k = 5, 100, 24, 12
    multi = oracle.OracleCache(U, L, B, k)
    single = [oracle.OracleCache(1, L, B, k) for _ in range(U)]
    for t in range(20):
        sel = np.stack([rng.choice(L, size=k, replace=False) for _ in range(U)]).astype(np.int32)
        slots, counts, pp, ps, bad = multi.resolve(sel)
        assert bad == 0
        for u in range(U):
            rc, s1, c1, p1, q1 = single[u].resolve_unit(0, sel[u])
            assert (s1 == slots[u]).all() and (c1 == counts[u]).all()
            m = int(c1[1])
            assert (p1 == pp[u, :m]).all() and (q1 == ps[u, :m]).all()


@pytest.mark.parametrize("bad", ["dup", "range", "dup_hit"])
def test_bad_selection_leaves_state_unchanged(bad):
    L, B, k = 50, 8, 4
    c = oracle.OracleCache(1, L, B, k)
    c.resolve_unit(0, np.array([1, 2, 3, 4]))
    before = (c.pt.copy(), c.slot_pos.copy(), c.slot_ts.copy(), c.clock.copy())
    sel = {"dup": [7, 9, 7, -1], "range": [7, 50, 3, 4], "dup_hit": [1, 1, 5, 6]}[bad]
    rc, slots, counts, pp, ps = c.resolve_unit(0, np.array(sel))
    assert rc == oracle.BAD_SELECTION
    assert (slots == -1).all() and counts.tolist() == [0, 0]
    for a, b in zip(before, (c.pt, c.slot_pos, c.slot_ts, c.clock)):
        assert (a == b).all()
    # a valid call afterwards proceeds with step clock 2
    rc, slots, counts, pp, ps = c.resolve_unit(0, np.array([1, 2, 3, 10]))
    assert rc == oracle.OK and counts.tolist() == [3, 1] and int(c.clock[0]) == 2


def test_padding_only_advances_clock():
    c = oracle.OracleCache(1, 10, 4, 3)
    rc, slots, counts, pp, ps = c.resolve_unit(0, np.array([-1, -1, -1]))
    assert rc == oracle.OK and slots.tolist() == [-1, -1, -1] and counts.tolist() == [0, 0]
    assert int(c.clock[0]) == 1 and (c.slot_pos == -1).all()


def test_apply_plan_copies_records():
    rng = np.random.default_rng(5)
    host = rng.integers(0, 255, size=(40, 48), dtype=np.uint8)
    cache = np.zeros((8, 48), dtype=np.uint8)
    c = oracle.OracleCache(1, 40, 8, 5)
    for t in range(10):
        sel = rng.choice(40, size=5, replace=False).astype(np.int32)
        rc, slots, counts, pp, ps = c.resolve_unit(0, sel)
        oracle.apply_plan(host, cache, pp, ps)
        assert (cache[slots] == host[sel]).all()
        res = np.nonzero(c.slot_pos[0] >= 0)[0]
        assert (cache[res] == host[c.slot_pos[0][res]]).all()


def test_admission_worked_example():
    """Write-through admission (Section 3.3 (4)) as a one-entry resolve event, by hand: B = 3,
    k = 2, cold start. Step 1 [9, 5]: misses 5 -> slot 0, 9 -> slot 1 (stamp 1). Admit 12
    (event 2): the empty slot 2 (stamp 0) is least recent -> 12 -> 2, stamp 3. Step 3 [12, 7]:
    12 hits slot 2 (stamp 6); 7 misses and takes the least recent non-hit slot, 0 (stamp 1, tie
    with slot 1 broken by slot), evicting 5. Admit 13 (event 4): slot 1 (9, stamp 1) is least
    recent -> 13 -> 1. Admit 7 (event 5): resident, refreshed in place."""
    c = oracle.OracleCache(1, 16, 3, 2)
    rc, slots, counts, _, _ = c.resolve_unit(0, np.array([9, 5]))
    assert rc == oracle.OK and slots.tolist() == [1, 0]
    assert c.admit_unit(0, 12) == (oracle.OK, 2, False)
    assert c.slot_ts[0].tolist() == [1, 1, 3]
    rc, slots, counts, _, _ = c.resolve_unit(0, np.array([12, 7]))
    assert slots.tolist() == [2, 0] and counts.tolist() == [1, 1]
    assert c.pt[0, 5] == -1
    assert c.admit_unit(0, 13) == (oracle.OK, 1, False)
    assert c.pt[0, 9] == -1 and c.slot_pos[0].tolist() == [7, 13, 12]
    assert c.admit_unit(0, 7) == (oracle.OK, 0, True)
    assert c.slot_ts[0].tolist() == [10, 7, 6] and int(c.clock[0]) == 5
    assert c.admit_unit(0, 16)[0] == oracle.BAD_SELECTION  # outside [0, L): state unchanged
    assert int(c.clock[0]) == 5


@pytest.mark.parametrize("seed", range(4))
def test_admission_matches_list_lru(seed):
    """Resolve steps interleaved with admissions agree with the independent list model, where an
    admission is an access of the one-position set {p}; an admitted position is resident and,
    holding the newest stamp, survives until B other slots have been touched after it."""
    rng = np.random.default_rng(300 + seed)
    for trial in range(40):
        L = int(rng.integers(8, 64))
        B = int(rng.integers(2, 17))
        k = int(rng.integers(1, min(B, L) + 1))
        model = ListLRU(B)
        c = oracle.OracleCache(1, L, B, k)
        for t in range(int(rng.integers(2, 30))):
            if rng.random() < 0.4:
                p = int(rng.integers(0, L))
                rc, slot, was_hit = c.admit_unit(0, p)
                e_slots, e_counts, _ = model.step(np.array([p]))
                assert rc == oracle.OK and slot == e_slots[0]
                assert was_hit == (e_counts[0] == 1)
                assert c.pt[0, p] == slot and c.slot_pos[0, slot] == p
                assert c.slot_ts[0, slot] == c.slot_ts[0].max()
            else:
                sel = rng.choice(L, size=k, replace=False).astype(np.int32)
                rc, slots, counts, pp, ps = c.resolve_unit(0, sel)
                e_slots, e_counts, e_plan = model.step(sel)
                assert rc == oracle.OK and slots.tolist() == e_slots
                assert list(zip(pp.tolist(), ps.tolist())) == e_plan


@pytest.mark.parametrize("seed", range(3))
def test_request_readmission_is_a_cold_cache(seed):
    """Releasing a unit and admitting a new request into it (Section 3.3 (2)) starts that unit
    from the cold state: from then on it agrees with a fresh independent list model fed only
    the new request's selections, while the other units keep agreeing with the models that
    have seen their whole history."""
    rng = np.random.default_rng(400 + seed)
    for trial in range(20):
        U = 3
        L = int(rng.integers(8, 64))
        B = int(rng.integers(2, 17))
        k = int(rng.integers(1, min(B, L) + 1))
        models = [ListLRU(B) for _ in range(U)]
        c = oracle.OracleCache(U, L, B, k)
        steps = int(rng.integers(4, 30))
        swap = int(rng.integers(1, steps))
        victim = int(rng.integers(0, U))
        for t in range(steps):
            if t == swap:
                c.reset_unit(victim)
                models[victim] = ListLRU(B)
                assert (c.pt[victim] == -1).all() and (c.slot_pos[victim] == -1).all()
                assert c.clock[victim] == 0 and (c.slot_ts[victim] == 0).all()
            sel = np.stack([rng.choice(L, size=k, replace=False) for _ in range(U)])
            slots, counts, pp, ps, bad = c.resolve(sel.astype(np.int32))
            assert bad == 0
            for u in range(U):
                e_slots, e_counts, e_plan = models[u].step(sel[u])
                assert slots[u].tolist() == e_slots, (trial, t, u)
                assert counts[u].tolist() == list(e_counts)
                m = int(counts[u][1])
                assert list(zip(pp[u][:m].tolist(), ps[u][:m].tolist())) == e_plan
