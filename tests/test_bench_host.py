"""Host logic of the benchmark (no GPU): the busy time of overlapping transfer intervals, the
lookup of counter-measured traffic, which must return nothing once a kernel's source differs
from the one the counters were taken on, the threaded CPU baseline, and the default run's child
process per workload."""
import os

import numpy as np
import pytest

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
    # a record that names an attention plan applies to that plan only
    b.write_bytes(b"#pragma once\n")
    with open(tmp_path / "profiles" / "k.md", "a") as f:
        f.write(f"traffic-record workload=w1 kernel=sparse_decode plan=own-gpu source=src/k.hip,src/k.h "
                f"sha256={sha} fetch_bytes=7 write_bytes=8\n")
    assert bench.traffic_record("w1", "sparse_decode", "own-gpu")["write_bytes"] == 8
    assert bench.traffic_record("w1", "sparse_decode", "beside-fetch") is None
    assert bench.traffic_record("w1", "sparse_decode") is None


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
    assert 0 < r["whole_step_selections_per_s"] < r["value"]


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


class _FakeHip:
    """Events and streams as integers; every record and wait is logged and checked: no use of
    a destroyed event, no wait on an event that was never recorded."""

    def __init__(self):
        self.next, self.live, self.recorded, self.log = 1000, set(), set(), []

    def event(self):
        self.next += 1
        self.live.add(self.next)
        return self.next

    def destroy(self, e):
        assert e in self.live, "event destroyed twice"
        self.live.discard(e)
        self.recorded.discard(e)

    def rec(self, e, stream):
        assert e in self.live, "record of a destroyed event"
        self.recorded.add(e)
        self.log.append(("rec", e, stream))
        return 0

    def wait(self, stream, e, flags):
        assert e in self.live, "wait on a destroyed event"
        assert e in self.recorded, "wait on an event never recorded"
        self.log.append(("wait", stream, e))
        return 0


class _FakeLib:
    def __init__(self, log, args_log=None):
        self._log, self._args = log, args_log

    def __getattr__(self, name):
        if not name.startswith("hisparse_"):
            raise AttributeError(name)

        def call(*args):
            self._log.append(("call", name, args[-1]))  # the stream is the last argument
            if self._args is not None:
                self._args.append((len(self._log) - 1, name, args))
            return 0
        return call


LINK_S = 55  # the shared link stream of the link-stream cases


def _schedule(hip, *, layers, G, n_mb, schedule, speculate, append, turns, share, steps,
              handover=0, link=False, dturns=None, turn_slots=1, args_log=None):
    from types import SimpleNamespace
    w = SimpleNamespace(num_layers=layers, record_bytes=1152)
    groups = [(a, list(range(a + 1, min(a + G, layers)))) for a in range(0, layers, G)]
    mbs = []
    for i in range(n_mb):
        base = 10_000 * (i + 1)
        mbs.append(SimpleNamespace(
            u0=4 * i, U=4, h=7 + i, main=100 + 2 * i, side=101 + 2 * i,
            q_p=[[base + 10 * v + l for l in range(layers)] for v in range(2)],
            sel_p=[[base + 1000 + 100 * t + l for l in range(layers)] for t in range(steps)],
            cnt_p=[[base + 5000 + 100 * t + l for l in range(layers)] for t in range(steps)],
            spec_p=[[base + 7000 + 100 * t + l for l in range(layers)] for t in range(steps)],
            pos_p=[base + 9000 + t for t in range(steps)],
            new_p=[base + 9500 + t for t in range(steps)],
            slot_p=[base + 200 + l for l in range(layers)],
            out_p=[base + 300 + l for l in range(layers)], ws_ptr=base + 400, ws_bytes=1 << 20,
            adm_ptr=base + 500, sync=[hip.event(), hip.event()],
            link=[hip.event() for _ in groups], rdone=[hip.event() for _ in groups]))
    return bench.DecodeSchedule(
        w=w, k=2048, groups=groups, mbs=mbs, n_mb=n_mb, n_qv=2, ad_ref=None,
        lib=_FakeLib(hip.log, args_log), rec=hip.rec, wait=hip.wait, root_s=1,
        fork_ev=hip.event(), join_evs=[hip.event() for _ in mbs], schedule=schedule, turns=turns,
        speculate=speculate, append=append, share=share, status_string=str, handover=handover,
        link_s=LINK_S if link else None, link_join=hip.event() if link else None, dturns=dturns,
        turn_slots=turn_slots, turn_share=192)


TRANSFERS = ("hisparse_fetch", "hisparse_fetch_group", "hisparse_fetch_part")


def test_decode_schedule_events_and_turns():
    """Every option of the benchmark's decode step, run through recorders: the timing events a
    step consumes stay within its budget and are distinct, no stream waits on an event that was
    destroyed or never recorded (warm-up steps without timing events, then timed steps whose
    events are destroyed after each step), and with turns taken at every layer each micro-batch's
    transfer waits for the previous transfer's event, in the order of groups and micro-batches."""
    cases = []
    for schedule in ("overlap", "serial", "side", "batched"):
        for n_mb in (1, 2, 3):
            cases.append(dict(layers=8, G=4, n_mb=n_mb, schedule=schedule, speculate=False,
                              append=False, turns="all", share=0))
    cases += [dict(layers=8, G=4, n_mb=2, schedule="overlap", speculate=False, append=True,
                   turns="first", share=64),
              dict(layers=6, G=1, n_mb=2, schedule="overlap", speculate=True, append=True,
                   turns="all", share=0),
              dict(layers=6, G=1, n_mb=1, schedule="overlap", speculate=True, append=False,
                   turns="all", share=0),
              dict(layers=61, G=4, n_mb=1, schedule="overlap", speculate=False, append=False,
                   turns="all", share=64),
              dict(layers=8, G=1, n_mb=2, schedule="overlap", speculate=False, append=True,
                   turns="all", share=0, handover=200),
              dict(layers=8, G=4, n_mb=3, schedule="side", speculate=False, append=False,
                   turns="all", share=0, handover=128),
              dict(layers=6, G=1, n_mb=2, schedule="overlap", speculate=True, append=False,
                   turns="all", share=0, handover=100)]
    steps = 6
    for case in cases:
        hip = _FakeHip()
        sched = _schedule(hip, steps=steps, **case)
        budget = sched.events_per_step()
        timing = set()
        for t in range(2):  # warm-up: no timing events
            sched.step(t)
        for t in range(2, steps):
            ev = [hip.event() for _ in range(budget)]
            given = list(ev)
            timing.update(given)
            spans = []
            sched.step(t, ev, spans)
            used = [e for _, e0, e1 in spans for e in (e0, e1)]
            assert len(used) == len(set(used)) <= budget, case
            assert set(used) <= set(given), case
            for e in given:  # the span pass keeps them longer; destroying early is stricter
                hip.destroy(e)
        # turns: each transfer after the first of a step waits for the previous transfer's
        # link event
        if case["n_mb"] > 1 and case["turns"] == "all":
            mbs = sched.mbs
            links = {e for mb in mbs for e in mb.link}
            log = [x for x in hip.log if not (x[0] == "rec" and x[1] in timing)]
            # a transfer that holds the link turn: followed by the record of a link event
            calls = [i for i, x in enumerate(log) if x[0] == "call" and x[1] in TRANSFERS and
                     log[i + 1][0] == "rec" and log[i + 1][1] in links]
            n_groups = len(sched.groups)
            per_step = n_groups * case["n_mb"]
            assert len(calls) == steps * per_step, case
            for j, i in enumerate(calls):
                g, m = divmod(j % per_step, case["n_mb"])
                assert log[i + 1] == ("rec", mbs[m].link[g], mbs[m].main), case
                if j % per_step:
                    pg, pm = divmod(j % per_step - 1, case["n_mb"])
                    assert log[i - 1] == ("wait", mbs[m].main, mbs[pm].link[pg]), case
                if case.get("handover"):  # the rest of the fetch after the turn passed on
                    assert log[i][1] == "hisparse_fetch_part", case
                    assert log[i + 2] == ("call", "hisparse_fetch_part", mbs[m].main), case


def test_decode_schedule_link_stream():
    """The shared link stream: every micro-batch's transfer goes to one stream in the order of
    groups and micro-batches, waits there for its own micro-batch's resolve (an event recorded
    on that micro-batch's stream right after the resolve), and is followed by the record of its
    link event, which the micro-batch's stream waits for before its attention. The link stream
    forks from the root stream with the micro-batches and joins back into it; no wait names a
    destroyed or never-recorded event, over single steps and over steps captured several to a
    graph (fork at the first, join at the last). Options it cannot combine with are refused."""
    cases = [dict(layers=8, G=1, n_mb=2, schedule="overlap", speculate=False, append=False),
             dict(layers=8, G=1, n_mb=3, schedule="overlap", speculate=False, append=True),
             dict(layers=6, G=1, n_mb=2, schedule="overlap", speculate=True, append=False),
             dict(layers=8, G=4, n_mb=2, schedule="serial", speculate=False, append=False),
             dict(layers=8, G=4, n_mb=2, schedule="overlap", speculate=False, append=False)]
    steps = 8
    for case in cases:
        hip = _FakeHip()
        sched = _schedule(hip, steps=steps, turns="all", share=0, link=True, **case)
        budget = sched.events_per_step()
        timing = set()
        sched.step(0)
        sched.step(1)
        for t0 in (2, 5):  # a graph of 3 steps, twice: fork at the first, join at the last
            for j in range(3):
                ev = [hip.event() for _ in range(budget)]
                timing.update(ev)
                spans = []
                sched.step(t0 + j, ev, spans, fork=(j == 0), join=(j == 2))
                used = [e for _, e0, e1 in spans for e in (e0, e1)]
                assert len(used) == len(set(used)) <= budget, case
                for e in ev:
                    hip.destroy(e)
        mbs, n_mb = sched.mbs, case["n_mb"]
        log = [x for x in hip.log if not (x[0] == "rec" and x[1] in timing)]
        calls = [i for i, x in enumerate(log) if x[0] == "call" and x[1] in TRANSFERS]
        per_step = len(sched.groups) * n_mb
        assert len(calls) == steps * per_step, case
        for j, i in enumerate(calls):
            g, m = divmod(j % per_step, n_mb)
            mb = mbs[m]
            assert log[i][2] == LINK_S, case
            assert log[i - 2:i] == [("rec", mb.rdone[g], mb.main), ("wait", LINK_S, mb.rdone[g])]
            assert log[i + 1:i + 3] == [("rec", mb.link[g], LINK_S), ("wait", mb.main, mb.link[g])]
            # the resolve of that group precedes it on the micro-batch's stream
            prev = [x for x in log[:i - 2] if x[0] == "call" and x[2] == mb.main]
            assert prev[-1][1] == "hisparse_resolve_tables", case
        # no attention before its transfer: every attention call of a micro-batch follows the
        # wait for its latest link event on that stream
        for mb in mbs:
            waited = False
            for x in log:
                if x[0] == "rec" and x[1] in mb.rdone:  # a new transfer is on its way
                    waited = False
                if x[0] == "wait" and x[1] == mb.main and x[2] in mb.link:
                    waited = True
                if x[0] == "call" and x[2] == mb.main and "decode" in x[1]:
                    assert waited, case
        forks = [x for x in log if x == ("wait", LINK_S, sched.fork_ev)]
        joins = [i for i, x in enumerate(log) if x == ("rec", sched.link_join, LINK_S)]
        assert len(forks) == 2 + 2 and len(joins) == 2 + 2, case
        for i in joins:
            assert log[i + 1] == ("wait", 1, sched.link_join), case
    hip = _FakeHip()
    for bad in (dict(n_mb=1, turns="all", handover=0), dict(n_mb=2, turns="first", handover=0),
                dict(n_mb=2, turns="all", handover=64)):
        with pytest.raises(ValueError):
            _schedule(hip, layers=4, G=1, schedule="overlap", speculate=False, append=False,
                      share=0, steps=2, link=True, **bad)


DTURNS = 4242  # the device turn array of the device-turn cases


def test_decode_schedule_device_turns():
    """Link turns taken on the device: every micro-batch's transfer is a hisparse_fetch_turn on
    its own stream (no event between the micro-batches' streams for the link), waiting for the
    turn the previous transfer (in group and micro-batch order) signals, within one window of
    turns reset on the root stream before the fork that starts it (every step when enqueued
    one by one, the first of the steps captured to a graph). Turn indices stay inside the
    array, each is signalled once per window and waited for at most once, and only after its
    signalling call was enqueued. Options it cannot combine with are refused."""
    cases = [dict(layers=8, G=1, n_mb=2, schedule="overlap", speculate=False, append=False,
                  turns="all"),
             dict(layers=8, G=1, n_mb=3, schedule="overlap", speculate=False, append=True,
                  turns="all"),
             dict(layers=6, G=1, n_mb=2, schedule="overlap", speculate=True, append=False,
                  turns="all"),
             dict(layers=8, G=1, n_mb=2, schedule="overlap", speculate=False, append=False,
                  turns="first"),
             dict(layers=8, G=4, n_mb=2, schedule="overlap", speculate=False, append=False,
                  turns="all"),
             dict(layers=8, G=4, n_mb=2, schedule="side", speculate=False, append=False,
                  turns="all")]
    steps, S = 8, 3
    for case in cases:
        hip, args_log = _FakeHip(), []
        sched = _schedule(hip, steps=steps, share=0, dturns=DTURNS, turn_slots=S,
                          args_log=args_log, **case)
        budget = sched.events_per_step()
        windows = [[0], [1]]  # steps of each window of turns
        sched.step(0)
        sched.step(1)
        for t0 in (2, 5):  # a graph of 3 steps, twice: fork at the first, join at the last
            windows.append([t0, t0 + 1, t0 + 2])
            for j in range(S):
                ev = [hip.event() for _ in range(budget)]
                sched.step(t0 + j, ev, [], fork=(j == 0), join=(j == S - 1))
                for e in ev:
                    hip.destroy(e)
        mbs, n_mb, n_groups = sched.mbs, case["n_mb"], len(sched.groups)
        n_turns = S * n_groups * n_mb
        assert sched.n_turns() == n_turns
        streams = {mb.main: i for i, mb in enumerate(mbs)}
        links = {e for mb in mbs for e in mb.link}
        assert not [x for x in hip.log if x[0] == "wait" and x[2] in links], case
        ordered = n_groups if case["turns"] == "all" else 1  # groups that take turns
        plain = [a for a in args_log if a[1] in TRANSFERS]
        assert len(plain) == steps * (n_groups - ordered) * n_mb, case
        assert all(a[1] == "hisparse_fetch" for a in plain), case
        resets = [a for a in args_log if a[1] == "hisparse_link_turns_reset"]
        fetches = [a for a in args_log if a[1] == "hisparse_fetch_turn"]
        # the eager steps 0 and 1 reset once each; each graph once
        assert len(resets) == 2 + 2, case
        for i, _, args in resets:
            assert args == (DTURNS, n_turns, 1), case
            assert hip.log[i + 1] == ("rec", sched.fork_ev, 1), case  # before the fork
        assert len(fetches) == steps * ordered * n_mb, case
        bounds = [i for i, _, _ in resets] + [len(hip.log)]
        for w in range(len(resets)):  # one window of turns
            win = [f for f in fetches if bounds[w] < f[0] < bounds[w + 1]]
            signalled = set()
            chain = []
            for i, _, args in win:
                h, layer, dt, nt, wt, sg, share, stream = args
                assert dt == DTURNS and nt == n_turns, case
                assert share == 192 and stream in streams, case
                assert 0 <= sg < n_turns and sg not in signalled, case
                assert wt == -1 or (0 <= wt < n_turns and wt in signalled), case
                signalled.add(sg)
                chain.append((wt, sg, streams[stream]))
            # within each step of the window: transfers in group-major, micro-batch order,
            # each (after the first of the step) waiting for the one before it
            per_step = ordered * n_mb
            assert len(chain) == len(windows[w]) * per_step, case
            for q, (wt, sg, m) in enumerate(chain):
                j, r = divmod(q, per_step)
                g, i = divmod(r, n_mb)
                t = windows[w][j]
                assert m == i and sg == sched.turn_index(t, g, i), case
                assert wt == (chain[q - 1][1] if r else -1), case
            # each micro-batch's transfer follows its own resolve on its stream
        for i, name, args in fetches:
            prev = [x for x in hip.log[:i] if x[0] == "call" and x[2] == args[-1]]
            assert prev[-1][1] == "hisparse_resolve_tables", case
    hip = _FakeHip()
    for bad in (dict(n_mb=1, schedule="overlap"), dict(n_mb=2, schedule="overlap", handover=64),
                dict(n_mb=2, schedule="serial", G=4), dict(n_mb=2, schedule="overlap", link=True)):
        bad.setdefault("G", 1)
        with pytest.raises(ValueError):
            _schedule(hip, layers=4, speculate=False, append=False, turns="all", share=0,
                      steps=2, dturns=DTURNS, **bad)
