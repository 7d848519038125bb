"""GPU parity of the resolve path (Section 3.4 phases 1-5) against the CPU oracle.

Bit-exact on every step: the slot vector of every unit, (hits, misses), and the miss plan;
at checkpoints: the full LRU state (slot map, timestamps, page table, clock, recency index)
and the bytes of every resident slot against the host record it claims to hold."""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, expected_order, layer_cache_host, log, turn_step
from paper_2608_07009_amd import HiSparseCache, hisparse as hs

pytestmark = pytest.mark.gpu

# full shapes; steps trimmed so every config finishes in well under a minute
STEPS = {1: 64, 2: 40, 3: 128, 4: 64, 5: 24}


def check_state(run, layer, orc, full_pt=True):
    st = run.cache.read_state(layer, page_table=full_pt)
    assert (st["slot_pos"] == orc.slot_pos).all()
    assert (st["slot_ts"] == orc.slot_ts).all()
    assert (st["clock"] == orc.clock).all()
    assert (st["order"] == expected_order(orc.slot_ts)).all()
    if full_pt:
        assert (st["page_table"] == orc.pt).all()


def check_resident_bytes(run, layer, orc):
    """Every resident slot holds exactly the host record its slot map names."""
    img = layer_cache_host(run, layer)
    host = run.cache.host_view(layer)
    for u in range(run.w.units):
        res = np.nonzero(orc.slot_pos[u] >= 0)[0]
        assert (img[u, res] == host[u, orc.slot_pos[u, res]]).all(), f"unit {u}"


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_resolve_matches_oracle(cfg):
    steps = STEPS[cfg]
    log(f"test_resolve_matches_oracle cfg={cfg} steps={steps}")
    run = Run(W.workload(cfg), steps)
    w = run.w
    try:
        orcs = {l: oracle.OracleCache(w.units, w.L, w.B, w.k) for l in w.anchors}
        checkpoints = {0, 1, steps // 2, steps - 1}
        for t in range(steps):
            run.resolve_step(t)
            slots = run.slots.cpu().numpy()
            counts = run.counts.cpu().numpy()
            for l in w.anchors:
                a = l // w.share_group
                sel = run.sel_host[t, a * w.units:(a + 1) * w.units]
                e_slots, e_counts, pp, ps, bad = orcs[l].resolve(sel)
                assert bad == 0
                assert (slots[l] == e_slots).all(), f"slots step {t} layer {l}"
                assert (counts[l] == e_counts).all(), f"counts step {t} layer {l}"
                if t in checkpoints and l in (w.anchors[0], w.anchors[-1]):
                    plan, cnt = run.cache.read_plan(l)
                    assert (cnt == e_counts[:, 1]).all()
                    for u in range(w.units):
                        m = cnt[u]
                        assert (plan[u, :m, 0] == pp[u, :m]).all()
                        assert (plan[u, :m, 1] == ps[u, :m]).all()
                    check_state(run, l, orcs[l], full_pt=(w.units * w.L <= 1 << 24))
                    check_resident_bytes(run, l, orcs[l])
            if t in checkpoints:
                log(f"  step {t}: hits/misses unit0 layer0 = {counts[0, 0].tolist()}")
        st, info = run.cache.check_errors()
        assert st == hs.HISPARSE_OK
    finally:
        run.close()


def test_resolve_fetch_none_same_tables():
    """FETCH_NONE (no-IO timing mode) publishes the same slot tables and counts."""
    w = W.workload(1)
    a = Run(w, 32)
    b = Run(w, 32, fill=False, fetch=hs.HISPARSE_FETCH_NONE)
    try:
        for t in range(32):
            a.resolve_step(t)
            b.resolve_step(t)
            assert torch.equal(a.slots, b.slots) and torch.equal(a.counts, b.counts)
    finally:
        a.close()
        b.close()


@pytest.mark.parametrize("cfg,steps,fetch", [(1, 24, hs.HISPARSE_FETCH_SDMA),
                                             (3, 24, hs.HISPARSE_FETCH_SDMA),
                                             (1, 24, hs.HISPARSE_FETCH_STAGED),
                                             (2, 6, hs.HISPARSE_FETCH_STAGED),
                                             (3, 24, hs.HISPARSE_FETCH_STAGED),
                                             (4, 6, hs.HISPARSE_FETCH_STAGED)])
def test_host_issued_fetch_matches_zero_copy(cfg, steps, fetch):
    """The host-issued fetch paths (per-run copy-engine copies; host-gathered staging, one
    copy and a device scatter) move exactly the bytes the zero-copy kernel moves, and the
    resident bytes equal the oracle's host records."""
    w = W.workload(cfg, num_layers=1, num_requests=min(W.workload(cfg).num_requests, 4))
    a = Run(w, steps)
    b = Run(w, steps, fetch=fetch)
    orc = oracle.OracleCache(w.units, w.L, w.B, w.k)
    try:
        for t in range(steps):
            a.resolve_step(t)
            b.resolve_step(t)
            assert torch.equal(a.slots, b.slots) and torch.equal(a.counts, b.counts)
            orc.resolve(b.sel_host[t, :w.units])
            if t in (0, steps // 2, steps - 1):
                assert (layer_cache_host(a, 0) == layer_cache_host(b, 0)).all(), f"step {t}"
                check_resident_bytes(b, 0, orc)
    finally:
        a.close()
        b.close()


def test_resolve_padding_and_bad_selections():
    """Padding entries, repeated entries (resident and not) and out-of-range positions, on the
    device: bad units keep their state, publish -1 slots and (0, 0) counts, and the first error
    is latched; every other unit stays bit-exact with the oracle throughout."""
    U, L, B, k, steps = 4, 4096, 256, 96, 12
    rng = np.random.default_rng(20261202)
    dev = torch.device("cuda:0")
    cache = HiSparseCache(num_requests=U, num_layers=1, units_per_request=1, capacity=B,
                          num_records=L, top_k=k, record_bytes=64, fetch=hs.HISPARSE_FETCH_NONE)
    orc = oracle.OracleCache(U, L, B, k)
    slots = torch.empty((U, k), dtype=torch.int32, device=dev)
    counts = torch.empty((U, 2), dtype=torch.int32, device=dev)
    prev = None
    injected = []
    try:
        for t in range(steps):
            # a drifting window keeps some entries resident from step to step
            sel = np.stack([rng.choice(np.arange(64 * t, 64 * t + 400), size=k, replace=False)
                            for _ in range(U)]).astype(np.int32)
            sel[1, 5:15] = -1                           # padding in every step
            if t == 3:
                sel[0, 7] = sel[0, 8]                   # repeated entry
                injected.append((t, 0))
            if t == 5 and prev is not None:
                sel[2, :2] = prev[2, 0]                 # repeated entry resident from last step
                injected.append((t, 2))
            if t == 7:
                sel[3, 40] = L + 5                      # beyond the records
                injected.append((t, 3))
            sel_d = torch.from_numpy(sel).to(dev)
            hs.hisparse_resolve_tables(cache.handle, 0, sel_d, slots, counts,
                                       torch.cuda.current_stream())
            e_slots, e_counts, _, _, n_bad = orc.resolve(sel)
            got_s, got_c = slots.cpu().numpy(), counts.cpu().numpy()
            assert (got_s == e_slots).all(), f"slots step {t}"
            assert (got_c == e_counts).all(), f"counts step {t}"
            for (ti, u) in injected:
                if ti == t:
                    assert n_bad >= 1 and (got_s[u] == -1).all() and (got_c[u] == 0).all()
            prev = sel
        st = cache.read_state(0)
        assert (st["slot_pos"] == orc.slot_pos).all() and (st["slot_ts"] == orc.slot_ts).all()
        assert (st["page_table"] == orc.pt).all() and (st["clock"] == orc.clock).all()
        code, info = cache.check_errors()
        assert code == hs.HISPARSE_ERR_BAD_SELECTION
        assert info[0] == 0 and info[1] == 0     # first latched error: layer 0, unit 0 (step 3)
        assert info[2] == len(injected)
    finally:
        cache.close()


def test_fetch_units_ranges_equal_whole_fetch():
    """Phase 4 over disjoint unit ranges (ragged, one empty) leaves every slot of every unit
    byte-identical to one whole-layer fetch; ranges outside [0, units) are argument errors."""
    w = W.workload(3, num_layers=1)
    steps = 6
    log(f"test_fetch_units_ranges_equal_whole_fetch {w.name} units={w.units}")
    whole = Run(w, steps)
    parts = Run(w, steps)
    try:
        ranges = [(0, 5), (5, 0), (5, 25), (30, w.units - 30)]
        for t in range(steps):
            hs.hisparse_resolve_tables(whole.cache.handle, 0, whole.sel_ptr(t, 0), whole.slots[0],
                                       whole.counts[0], whole.stream)
            hs.hisparse_fetch(whole.cache.handle, 0, whole.stream)
            hs.hisparse_resolve_tables(parts.cache.handle, 0, parts.sel_ptr(t, 0), parts.slots[0],
                                       parts.counts[0], parts.stream)
            for u0, n in ranges:
                hs.hisparse_fetch_units(parts.cache.handle, 0, u0, n, parts.stream)
        assert torch.equal(whole.slots, parts.slots)
        a, b = layer_cache_host(whole, 0), layer_cache_host(parts, 0)
        orc_state = whole.cache.read_state(0, page_table=False)
        for u in range(w.units):
            res = np.nonzero(orc_state["slot_pos"][u] >= 0)[0]
            assert (a[u, res] == b[u, res]).all(), f"unit {u}"
        for u0, n in [(-1, 2), (0, w.units + 1), (w.units, 1)]:
            with pytest.raises(hs.HisparseError):
                hs.hisparse_fetch_units(parts.cache.handle, 0, u0, n, parts.stream)
    finally:
        whole.close()
        parts.close()


def clustered_streams(L, k, rng):
    """Selections whose misses cluster in position: a cold contiguous window, a contiguous run
    mixed with scattered draws and hits, two runs at opposite ends of the range (some rank
    bucket over the whole range then holds far more misses than the counting pass takes: the
    kernel sorts them), uniform draws, and a shorter run among draws. Unit 1 repeats one entry
    of its far-apart runs at step 2 (a bad selection found by the sort)."""
    steps = []
    w0 = np.arange(L - k, L)
    steps.append([w0, w0.copy()])
    run = np.arange(L // 2, L // 2 + k // 2)
    steps.append([np.concatenate([run, rng.choice(w0, k - k // 2, replace=False)])] * 2)
    far = np.concatenate([np.arange(0, k // 2), np.arange(L - 4096 - k // 2, L - 4096)])
    bad = far.copy()
    bad[7] = bad[k // 2 + 9]  # a repeated position, one in each run's place
    steps.append([far, bad])
    steps.append([rng.choice(L, k, replace=False)] * 2)
    short = np.arange(L // 3, L // 3 + 600)
    rest = rng.choice(np.setdiff1d(rng.choice(L, 4 * k, replace=False), short), k - 600,
                      replace=False)
    steps.append([np.concatenate([short, rest])] * 2)
    out = np.empty((len(steps), 2, k), dtype=np.int32)
    for t, per_unit in enumerate(steps):
        for u in range(2):
            out[t, u] = rng.permutation(np.asarray(per_unit[u], dtype=np.int64))
    return out


def test_resolve_clustered_misses_at_large_context():
    """2^24 records per unit, k = 2048, B = 4096: misses in contiguous runs (the rank buckets
    follow the misses' own position range; far-apart runs are sorted instead of counted) give
    the oracle's slots, counts, plans and tables bit for bit, and a repeated entry is still
    caught."""
    L, k, B = 1 << 24, 2048, 4096
    rng = np.random.default_rng(24)
    sel = clustered_streams(L, k, rng)
    log(f"test_resolve_clustered_misses_at_large_context L={L} k={k} B={B}")
    cache = HiSparseCache(num_requests=2, num_layers=1, units_per_request=1, capacity=B,
                          num_records=L, top_k=k, record_bytes=16)
    try:
        dev = torch.device("cuda:0")
        stream = torch.cuda.current_stream()
        host = cache.host_view(0)
        host[:] = rng.integers(0, 256, host.shape, dtype=np.uint8)
        orc = oracle.OracleCache(2, L, B, k)
        slots = torch.empty((2, k), dtype=torch.int32, device=dev)
        counts = torch.empty((2, 2), dtype=torch.int32, device=dev)
        for t in range(sel.shape[0]):
            sel_d = torch.from_numpy(sel[t]).to(dev)
            hs.hisparse_resolve(cache.handle, 0, sel_d, slots, counts, stream)
            e_slots, e_counts, pp, ps, n_bad = orc.resolve(sel[t])
            assert n_bad == (1 if t == 2 else 0)
            assert (slots.cpu().numpy() == e_slots).all(), f"slots step {t}"
            assert (counts.cpu().numpy() == e_counts).all(), f"counts step {t}"
            plan, count = cache.read_plan(0)
            for u in range(2):
                m = int(e_counts[u, 1])
                assert count[u] == m
                assert (plan[u, :m, 0] == pp[u, :m]).all() and (plan[u, :m, 1] == ps[u, :m]).all()
            st = cache.read_state(0, page_table=False)
            assert (st["slot_pos"] == orc.slot_pos).all() and (st["slot_ts"] == orc.slot_ts).all()
            assert (st["order"] == expected_order(orc.slot_ts)).all()
            status, info = cache.check_errors()
            if t == 2:
                assert status == hs.HISPARSE_ERR_BAD_SELECTION and list(info[:3]) == [0, 1, 1]
            else:
                assert status == hs.HISPARSE_OK
        st = cache.read_state(0)
        assert (st["page_table"] == orc.pt).all()
        img = d2h_cache(cache, 0).reshape(2, B, 16)
        for u in range(2):
            res = np.nonzero(orc.slot_pos[u] >= 0)[0]
            assert (img[u, res] == host[u, orc.slot_pos[u, res]]).all()
    finally:
        torch.cuda.synchronize()
        cache.close()


def d2h_cache(cache, layer):
    from hs_harness import d2h
    ptr, n = cache.layer_cache(layer)
    return d2h(ptr, n)


@pytest.mark.parametrize("fetch", [hs.HISPARSE_FETCH_SDMA, hs.HISPARSE_FETCH_STAGED])
def test_host_issued_fetch_refused_under_capture(fetch):
    """The host-issued fetch paths read the plan back with a synchronisation, so a fetch enqueued
    while the stream is capturing a HIP graph is refused (nothing is enqueued), and the same
    call works eagerly afterwards."""
    w = W.workload(1, num_layers=1)
    run = Run(w, 1, fetch=fetch)
    try:
        run.resolve_step(0)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        err = None
        with torch.cuda.graph(g, stream=s):
            try:
                hs.hisparse_fetch(run.cache.handle, 0, s)
            except hs.HisparseError as e:
                err = e
        assert err is not None and err.status == hs.HISPARSE_ERR_UNSUPPORTED
        hs.hisparse_fetch(run.cache.handle, 0, run.stream)
        torch.cuda.synchronize()
    finally:
        torch.cuda.synchronize()
        run.close()


@pytest.mark.parametrize("fetch", [hs.HISPARSE_FETCH_ZERO_COPY, hs.HISPARSE_FETCH_STAGED])
def test_fetch_parts_equal_fetch(fetch):
    """hisparse_fetch_part over adjacent plan ranges moves exactly what hisparse_fetch moves
    (every resident slot holds its host record); bad ranges are argument errors."""
    w = W.workload(2, num_requests=3, num_layers=1)
    steps = 4
    a, b = Run(w, steps), Run(w, steps, fetch=fetch)
    try:
        for t in range(steps):
            a.resolve_step(t)
            hs.hisparse_resolve_tables(b.cache.handle, 0, b.sel_ptr(t, 0), b.slots[0],
                                       b.counts[0], b.stream)
            cuts = [0, 37 + 40 * t, 200, 256]
            for lo, hi in zip(cuts[:-1], cuts[1:]):
                hs.hisparse_fetch_part(b.cache.handle, 0, lo, hi, b.stream)
            torch.cuda.synchronize()
            assert torch.equal(a.slots, b.slots) and torch.equal(a.counts, b.counts)
            assert (layer_cache_host(a, 0) == layer_cache_host(b, 0)).all(), f"step {t}"
        for lo, hi in ((-1, 10), (20, 10), (0, 300)):
            with pytest.raises(hs.HisparseError):
                hs.hisparse_fetch_part(b.cache.handle, 0, lo, hi, b.stream)
    finally:
        torch.cuda.synchronize()
        a.close()
        b.close()


def test_staged_fetches_on_two_streams():
    """The staged fetch path's buffers belong to the handle: an anchor's demand fetch on one
    stream and the replay of its plan into the shared layer on another, enqueued back to back
    with only the resolve ordered before both, each land exactly the planned records (the
    second call waits on the host for the first one's scatter before refilling the buffers)."""
    w = W.workload(2, num_requests=4, num_layers=2, share_group=2)
    steps = 4
    run = Run(w, steps, fetch=hs.HISPARSE_FETCH_STAGED)
    orc = oracle.OracleCache(w.units, w.L, w.B, w.k)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        for t in range(steps):
            log(f"staged two streams step {t}")
            with torch.cuda.stream(s1):
                hs.hisparse_resolve_tables(run.cache.handle, 0, run.sel_ptr(t, 0), run.slots[0],
                                           run.counts[0], s1)
                ev = torch.cuda.Event()
                ev.record(s1)
                hs.hisparse_fetch(run.cache.handle, 0, s1)
            s2.wait_event(ev)
            hs.hisparse_prefetch_layer(run.cache.handle, 0, 1, s2)
            torch.cuda.synchronize()
            orc.resolve(run.sel_host[t, :w.units])
            for layer in (0, 1):
                img = layer_cache_host(run, layer)
                host = run.cache.host_view(layer)
                for u in range(w.units):
                    res = np.nonzero(orc.slot_pos[u] >= 0)[0]
                    assert (img[u, res] == host[u, orc.slot_pos[u, res]]).all(), (t, layer, u)
    finally:
        run.close()


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_fetch_turns_on_two_streams_equal_fetch(cfg):
    """Two micro-batches (two caches, two streams) taking turns on the host link on the device
    (hisparse_fetch_turn, each transfer waiting for the previous one's signal): slots, counts and
    every layer's cache byte-identical to hisparse_resolve on a twin cache, every step; a turn
    that is never signalled only delays its launch (the wait ends by itself, after about 50 us
    when the signalling launch never started, about 4 ms when it did) and changes nothing; argument errors and the unsupported fetch paths are refused."""
    w = W.workload(cfg, num_requests=2, num_layers=2)
    steps = 4
    log(f"test_fetch_turns_on_two_streams_equal_fetch {w.name}")
    runs = [Run(w, steps), Run(w, steps)]
    twins = [Run(w, steps), Run(w, steps)]
    none = Run(w, 1, fill=False, fetch=hs.HISPARSE_FETCH_NONE)
    dev = runs[0].dev
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    n_turns = w.num_layers * len(runs)
    turns = torch.zeros(2 * n_turns, dtype=torch.int32, device=dev)
    try:
        torch.cuda.synchronize()
        for t in range(steps):
            log(f"fetch turns step {t}")
            turn_step(runs, streams, turns, t, w.num_layers)
            for r in twins:
                r.resolve_step(t)
            torch.cuda.synchronize()
            for r, tw in zip(runs, twins):
                assert torch.equal(r.slots, tw.slots) and torch.equal(r.counts, tw.counts), t
                for l in range(w.num_layers):
                    assert (layer_cache_host(r, l) == layer_cache_host(tw, l)).all(), (t, l)
            # every turn was signalled by all of its launch's workgroups
            tv = turns.view(n_turns, 2).cpu()
            assert (tv[:, 1] == 2).all() and (tv[:, 0] > 0).all(), tv
        # waits on turns never signalled: one whose launch never started (just reset) ends
        # after the start bound, one marked started from the host after the full bound; the
        # copies are the same
        s = streams[0]
        r, tw = runs[0], twins[0]
        for started, lo, hi in ((0, 0.04, 2.0), (1, 3.0, 1000.0)):
            hs.hisparse_link_turns_reset(turns, n_turns, s)
            with torch.cuda.stream(s):
                turns[3].fill_(started)  # turn 1's state word
            hs.hisparse_resolve_tables(r.cache.handle, 0, r.sel_ptr(started, 0), r.slots[0],
                                       r.counts[0], s)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            hs.hisparse_fetch_turn(r.cache.handle, 0, turns, n_turns, 1, 0, 256, s)
            e1.record(s)
            hs.hisparse_resolve(tw.cache.handle, 0, tw.sel_ptr(started, 0), tw.slots[0],
                                tw.counts[0], tw.stream)
            torch.cuda.synchronize()
            waited = e0.elapsed_time(e1)
            log(f"fetch waiting on an unsignalled turn (state {started}): {waited:.3f} ms")
            assert lo <= waited <= hi, (started, waited)
            assert torch.equal(r.slots[0], tw.slots[0]) and torch.equal(r.counts[0],
                                                                        tw.counts[0])
            assert (layer_cache_host(r, 0) == layer_cache_host(tw, 0)).all()
            assert int(turns[1].item()) == 2  # turn 0 signalled by the launch
        h = r.cache.handle
        N = n_turns
        for bad in ((h, 0, turns, N, 2, 2, 256), (h, 0, turns, N, -2, 0, 256),
                    (h, 0, turns, N, 0, 1, 0), (h, 0, turns, N, 0, 1, 257),
                    (h, 0, None, N, 0, 1, 256), (h, 0, turns, 0, -1, -1, 256),
                    (h, 0, turns, N, N, 0, 256), (h, 0, turns, N, 0, N, 256)):
            with pytest.raises(hs.HisparseError) as e:
                hs.hisparse_fetch_turn(*bad, s)
            assert e.value.status == hs.HISPARSE_ERR_INVALID_ARG, bad
        with pytest.raises(hs.HisparseError) as e:
            hs.hisparse_fetch_turn(none.cache.handle, 0, turns, N, -1, 0, 256, s)
        assert e.value.status == hs.HISPARSE_ERR_UNSUPPORTED
        for n in (0, 1 << 25):
            with pytest.raises(hs.HisparseError) as e:
                hs.hisparse_link_turns_reset(turns, n, s)
            assert e.value.status == hs.HISPARSE_ERR_INVALID_ARG
        torch.cuda.synchronize()
    finally:
        torch.cuda.synchronize()
        for r in runs + twins + [none]:
            r.close()
