"""HIP-graph capture of a whole decode step.

The paper captures resolve inside the decode graph, which requires every metadata update and IO
issue to replay without host-side branching (Appendix A, "Graph capture"). One step -- stage the
step's selection and query from a device-side step counter, then resolve + fetch + attention
for every layer -- is captured once and replayed for many steps. Each replay is checked against
an eager run of the same steps (slots, counts and attention outputs bit-identical), with eager
work and synchronisations between replays."""
import numpy as np
import pytest
import torch

import workload as W
from hs_harness import Run, attn_desc, layer_cache_host, log, turn_step
from paper_2608_07009_amd import hisparse as hs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg,layers,steps", [(1, 3, 12), (2, 2, 6)])
def test_graph_replay_matches_eager(cfg, layers, steps):
    w = W.workload(cfg, num_layers=layers)
    log(f"test_graph_replay_matches_eager {w.name} layers={layers} steps={steps}")
    eager = Run(w, steps)
    graph = Run(w, steps)
    try:
        dev = eager.dev
        ad = attn_desc(w)
        ws_bytes = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad)
        q_all = torch.stack([torch.stack([torch.from_numpy(W.queries(w, t, l).view(np.int16))
                                          for l in range(layers)]) for t in range(steps)]).to(dev)

        # eager reference
        ws_e = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        out_e = torch.empty((layers, w.units, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
        ref = []
        for t in range(steps):
            for l in range(layers):
                hs.hisparse_resolve(eager.cache.handle, l, eager.sel_ptr(t, l), eager.slots[l],
                                    eager.counts[l], eager.stream)
                hs.hisparse_sparse_decode(eager.cache.handle, l, q_all[t, l], eager.slots[l],
                                          out_e[l], ad, ws_e, ws_bytes, eager.stream)
            ref.append((eager.slots.clone(), eager.counts.clone(), out_e.clone()))
        torch.cuda.synchronize()

        # captured step
        ws_g = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        out_g = torch.empty_like(out_e)
        step = torch.zeros(1, dtype=torch.int64, device=dev)
        sel_buf = torch.empty_like(graph.sel[0])
        q_buf = torch.empty_like(q_all[0])
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                cs = torch.cuda.current_stream()
                sel_buf.copy_(graph.sel.index_select(0, step).squeeze(0))
                q_buf.copy_(q_all.index_select(0, step).squeeze(0))
                step.add_(1)
                for l in range(layers):
                    hs.hisparse_resolve(graph.cache.handle, l,
                                        sel_buf[l * w.units:(l + 1) * w.units], graph.slots[l],
                                        graph.counts[l], cs)
                    hs.hisparse_sparse_decode(graph.cache.handle, l, q_buf[l], graph.slots[l],
                                              out_g[l], ad, ws_g, ws_bytes, cs)
        torch.cuda.synchronize()
        for t in range(steps):
            g.replay()
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=dev).sum()  # eager work between replays
            e_slots, e_counts, e_out = ref[t]
            assert torch.equal(graph.slots, e_slots), f"slots differ at replay {t}"
            assert torch.equal(graph.counts, e_counts), f"counts differ at replay {t}"
            assert torch.equal(out_g, e_out), f"attention differs at replay {t}"
            del scratch
        st, _ = graph.cache.check_errors()
        assert st == hs.HISPARSE_OK
    finally:
        eager.close()
        graph.close()


def _shared_group_step(run, sel_ptr, q, out, ad, ws, ws_bytes, stream):
    """One decode step of a share group of 4 layers through every shared-layer entry point:
    resolve tables, fetch of the anchor by unit ranges, attention of layer 0 carrying the
    replay into layer 1, a multi-layer replay into layer 2, the group fetch (idempotent here),
    attention of layer 1, and layers 2-3 in one batched launch."""
    h, U = run.cache.handle, run.w.units
    hs.hisparse_resolve_tables(h, 0, sel_ptr, run.slots[0], run.counts[0], stream)
    hs.hisparse_fetch_units(h, 0, 0, 1, stream)
    hs.hisparse_fetch_units(h, 0, 1, U - 1, stream)
    hs.hisparse_sparse_decode_prefetch(h, 0, q[0], run.slots[0], out[0], ad, ws, ws_bytes,
                                       0, 1, 1, stream)
    hs.hisparse_prefetch_layers(h, 0, 2, 1, stream)
    hs.hisparse_fetch_group(h, 0, 4, stream)
    hs.hisparse_sparse_decode(h, 1, q[1], run.slots[0], out[1], ad, ws, ws_bytes, stream)
    hs.hisparse_sparse_decode_layers(h, 2, 2, q[2], run.slots[0], out[2], ad, ws, ws_bytes,
                                     stream)


def test_graph_replay_shared_layers():
    """The shared-layer entry points (unit-range fetch, replay carried by attention,
    multi-layer replay, group fetch, batched attention) replay from a captured graph with the
    same slots, counts, attention outputs and cache contents as eager calls."""
    w = W.workload(1, num_layers=4, share_group=4, num_requests=2)
    steps = 8
    log(f"test_graph_replay_shared_layers {w.name} steps={steps}")
    eager, graph = Run(w, steps), Run(w, steps)
    try:
        dev = eager.dev
        ad = attn_desc(w)
        ws_bytes = hs.hisparse_decode_workspace_bytes(2 * w.units, w.k, w.record_bytes, ad)
        q_all = torch.stack([torch.stack([torch.from_numpy(W.queries(w, t, l).view(np.int16))
                                          for l in range(4)]) for t in range(steps)]).to(dev)
        ws_e = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        out_e = torch.empty((4, w.units, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
        ref = []
        for t in range(steps):
            _shared_group_step(eager, eager.sel_ptr(t, 0), q_all[t], out_e, ad, ws_e, ws_bytes,
                               eager.stream)
            torch.cuda.synchronize()
            ref.append((eager.slots[0].clone(), eager.counts[0].clone(), out_e.clone(),
                        [layer_cache_host(eager, l) for l in range(4)]))

        ws_g = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        out_g = torch.empty_like(out_e)
        step = torch.zeros(1, dtype=torch.int64, device=dev)
        sel_buf = torch.empty_like(graph.sel[0])
        q_buf = torch.empty_like(q_all[0])
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                cs = torch.cuda.current_stream()
                sel_buf.copy_(graph.sel.index_select(0, step).squeeze(0))
                q_buf.copy_(q_all.index_select(0, step).squeeze(0))
                step.add_(1)
                _shared_group_step(graph, sel_buf[:w.units], q_buf, out_g, ad, ws_g, ws_bytes,
                                   cs)
        torch.cuda.synchronize()
        for t in range(steps):
            g.replay()
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=dev).sum()  # eager work between replays
            e_slots, e_counts, e_out, e_caches = ref[t]
            assert torch.equal(graph.slots[0], e_slots), f"slots differ at replay {t}"
            assert torch.equal(graph.counts[0], e_counts), f"counts differ at replay {t}"
            assert torch.equal(out_g, e_out), f"attention differs at replay {t}"
            for l in range(4):
                assert (layer_cache_host(graph, l) == e_caches[l]).all(), f"replay {t} layer {l}"
            del scratch
        assert graph.cache.check_errors()[0] == hs.HISPARSE_OK
    finally:
        eager.close()
        graph.close()


def test_graph_replay_append():
    """Resolve + fetch + write-through append captured in a graph: the appended position and
    record come from device buffers staged by the captured step itself; every replay matches
    the eager run (slots, admission slots, caches, and the host pools' appended records)."""
    steps = 8
    base = W.workload(1, num_layers=2, share_group=2, num_requests=2)
    L0 = base.L
    w = W.workload(1, num_layers=2, share_group=2, num_requests=2, L=L0 + steps)
    U, R = w.units, w.record_bytes
    log(f"test_graph_replay_append {w.name} steps={steps}")
    eager, graph = Run(w, steps, fill=False), Run(w, steps, fill=False)
    try:
        dev = eager.dev
        for r in (eager, graph):
            for l in range(2):
                r.cache.host_view(l)[:] = 0
                ptr = r.cache.host_pool(l)[0]
                for u in range(U):
                    W.fill_kv(ptr + u * w.L * R, base, l, u, 1)
        sel = torch.from_numpy(W.selection_streams(base, steps=steps)).to(dev)
        new = torch.from_numpy(np.stack([np.stack([np.stack(
            [W.kv_records(base, l, u, [L0 + t])[0] for u in range(U)]) for l in range(2)])
            for t in range(steps)]).view(np.int16)).to(dev)
        pos_e = torch.empty(U, dtype=torch.int32, device=dev)
        adm_e = torch.empty(U, dtype=torch.int32, device=dev)
        ref = []
        for t in range(steps):
            hs.hisparse_resolve(eager.cache.handle, 0, sel[t], eager.slots[0], eager.counts[0],
                                eager.stream)
            hs.hisparse_prefetch_layer(eager.cache.handle, 0, 1, eager.stream)
            pos_e.fill_(L0 + t)
            hs.hisparse_append(eager.cache.handle, 0, 2, pos_e, new[t], adm_e, eager.stream)
            torch.cuda.synchronize()
            ref.append((eager.slots[0].clone(), adm_e.clone(),
                        [layer_cache_host(eager, l) for l in range(2)]))

        step = torch.zeros(1, dtype=torch.int64, device=dev)
        sel_buf = torch.empty_like(sel[0])
        rec_buf = torch.empty_like(new[0])
        pos_buf = torch.empty(U, dtype=torch.int32, device=dev)
        adm_g = torch.empty(U, dtype=torch.int32, device=dev)
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                cs = torch.cuda.current_stream()
                sel_buf.copy_(sel.index_select(0, step).squeeze(0))
                rec_buf.copy_(new.index_select(0, step).squeeze(0))
                pos_buf.copy_((step + L0).to(torch.int32).expand(U))
                step.add_(1)
                hs.hisparse_resolve(graph.cache.handle, 0, sel_buf, graph.slots[0],
                                    graph.counts[0], cs)
                hs.hisparse_prefetch_layer(graph.cache.handle, 0, 1, cs)
                hs.hisparse_append(graph.cache.handle, 0, 2, pos_buf, rec_buf, adm_g, cs)
        torch.cuda.synchronize()
        for t in range(steps):
            g.replay()
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=dev).sum()  # eager work between replays
            e_slots, e_adm, e_caches = ref[t]
            assert torch.equal(graph.slots[0], e_slots), f"slots differ at replay {t}"
            assert torch.equal(adm_g, e_adm), f"admission slots differ at replay {t}"
            for l in range(2):
                assert (layer_cache_host(graph, l) == e_caches[l]).all(), f"replay {t} layer {l}"
            del scratch
        for l in range(2):
            a = eager.cache.host_view(l)[:, L0:]
            b = graph.cache.host_view(l)[:, L0:]
            assert (a == b).all() and (a != 0).any()
        assert graph.cache.check_errors()[0] == hs.HISPARSE_OK
    finally:
        torch.cuda.synchronize()
        eager.close()
        graph.close()


def test_graph_replay_lifecycle():
    """Request turnover captured in a graph: every replay releases unit 1's request (cold reset
    of its tables), stages a new request's records into unit 1's host pools from a device
    buffer picked by a device-side step counter, then resolves and fetches a step for both
    units. Every replay matches the eager run (slots, counts, tables, caches, host pools)."""
    steps = 4
    w = W.workload(1, num_layers=2, share_group=2, num_requests=2)
    U, L, R = w.units, w.L, w.record_bytes
    log(f"test_graph_replay_lifecycle {w.name} steps={steps}")
    eager, graph = Run(w, steps), Run(w, steps)
    try:
        dev = eager.dev
        srcs = np.empty((steps, 2, L, R), dtype=np.uint8)  # per replay: unit 1's new records
        for t in range(steps):
            wt = W.workload(1, num_layers=2, share_group=2, num_requests=2, seed=w.seed + 11 + t)
            for l in range(2):
                W.fill_kv(srcs[t, l].ctypes.data, wt, l, 1, 1)
        srcs_d = torch.from_numpy(srcs).to(dev)
        sel = eager.sel
        ref = []
        for t in range(steps):
            h = eager.cache.handle
            hs.hisparse_reset_units(h, 1, 1, eager.stream)
            hs.hisparse_stage(h, 0, 2, 1, 1, 0, L, srcs_d[t], L * R, eager.stream)
            hs.hisparse_resolve(h, 0, sel[t], eager.slots[0], eager.counts[0], eager.stream)
            hs.hisparse_prefetch_layer(h, 0, 1, eager.stream)
            torch.cuda.synchronize()
            ref.append((eager.slots[0].clone(), eager.counts[0].clone(),
                        eager.cache.read_state(0), [layer_cache_host(eager, l) for l in range(2)],
                        [eager.cache.host_view(l).copy() for l in range(2)]))

        step = torch.zeros(1, dtype=torch.int64, device=dev)
        sel_buf = torch.empty_like(sel[0])
        src_buf = torch.empty_like(srcs_d[0])
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                cs = torch.cuda.current_stream()
                sel_buf.copy_(sel.index_select(0, step).squeeze(0))
                src_buf.copy_(srcs_d.index_select(0, step).squeeze(0))
                step.add_(1)
                h = graph.cache.handle
                hs.hisparse_reset_units(h, 1, 1, cs)
                hs.hisparse_stage(h, 0, 2, 1, 1, 0, L, src_buf, L * R, cs)
                hs.hisparse_resolve(h, 0, sel_buf, graph.slots[0], graph.counts[0], cs)
                hs.hisparse_prefetch_layer(h, 0, 1, cs)
        torch.cuda.synchronize()
        for t in range(steps):
            g.replay()
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=dev).sum()  # eager work between replays
            e_slots, e_counts, e_st, e_caches, e_pools = ref[t]
            assert torch.equal(graph.slots[0], e_slots), f"slots differ at replay {t}"
            assert torch.equal(graph.counts[0], e_counts), f"counts differ at replay {t}"
            st = graph.cache.read_state(0)
            for key in ("slot_pos", "slot_ts", "order", "clock", "page_table"):
                assert (st[key] == e_st[key]).all(), f"{key} differs at replay {t}"
            for l in range(2):
                assert (layer_cache_host(graph, l) == e_caches[l]).all(), f"replay {t} layer {l}"
                assert (graph.cache.host_view(l) == e_pools[l]).all(), f"pool {t} layer {l}"
                assert (graph.cache.host_view(l)[1] == srcs[t, l]).all()
            del scratch
        assert graph.cache.check_errors()[0] == hs.HISPARSE_OK
    finally:
        torch.cuda.synchronize()
        eager.close()
        graph.close()


def test_graph_replay_speculate():
    """Resolve of layer 0, its selection as a hint for layer 1 (hisparse_speculate), resolve of
    layer 1, captured in a graph: every replay matches the eager run (slots, counts, hint
    counts, tables, caches)."""
    steps = 6
    w = W.workload(1, num_layers=2, share_group=1, num_requests=2)
    U = w.units
    log(f"test_graph_replay_speculate {w.name} steps={steps}")
    eager, graph = Run(w, steps), Run(w, steps)
    try:
        dev = eager.dev
        sel = torch.from_numpy(W.correlate_layers(w, eager.sel_host, 0.5, seed=5)).to(dev)
        hc_e = torch.empty((U, 2), dtype=torch.int32, device=dev)
        ref = []
        for t in range(steps):
            h = eager.cache.handle
            hs.hisparse_resolve(h, 0, sel[t, :U], eager.slots[0], eager.counts[0], eager.stream)
            hs.hisparse_speculate(h, 1, sel[t, :U], hc_e, eager.stream)
            hs.hisparse_resolve(h, 1, sel[t, U:], eager.slots[1], eager.counts[1], eager.stream)
            torch.cuda.synchronize()
            ref.append((eager.slots.clone(), eager.counts.clone(), hc_e.clone(),
                        eager.cache.read_state(1), [layer_cache_host(eager, l) for l in range(2)]))
        step = torch.zeros(1, dtype=torch.int64, device=dev)
        sel_buf = torch.empty_like(sel[0])
        hc_g = torch.empty((U, 2), dtype=torch.int32, device=dev)
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                cs = torch.cuda.current_stream()
                sel_buf.copy_(sel.index_select(0, step).squeeze(0))
                step.add_(1)
                h = graph.cache.handle
                hs.hisparse_resolve(h, 0, sel_buf[:U], graph.slots[0], graph.counts[0], cs)
                hs.hisparse_speculate(h, 1, sel_buf[:U], hc_g, cs)
                hs.hisparse_resolve(h, 1, sel_buf[U:], graph.slots[1], graph.counts[1], cs)
        torch.cuda.synchronize()
        for t in range(steps):
            g.replay()
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=dev).sum()  # eager work between replays
            e_slots, e_counts, e_hc, e_st, e_caches = ref[t]
            assert torch.equal(graph.slots, e_slots), f"slots differ at replay {t}"
            assert torch.equal(graph.counts, e_counts), f"counts differ at replay {t}"
            assert torch.equal(hc_g, e_hc), f"hint counts differ at replay {t}"
            st = graph.cache.read_state(1)
            for key in ("slot_pos", "slot_ts", "order", "clock", "page_table"):
                assert (st[key] == e_st[key]).all(), f"{key} differs at replay {t}"
            for l in range(2):
                assert (layer_cache_host(graph, l) == e_caches[l]).all(), f"replay {t} layer {l}"
            del scratch
        assert graph.cache.check_errors()[0] == hs.HISPARSE_OK
    finally:
        torch.cuda.synchronize()
        eager.close()
        graph.close()


def test_graph_replay_with_device_link_turns():
    """Two micro-batches taking device link turns, captured to a graph with the turns' reset
    (a fill kernel, no memset node) at its start, the micro-batches forked from and joined back
    into the capturing stream; every replay (eager work and synchronisations between them)
    leaves slots, counts and caches identical to hisparse_resolve on twin caches."""
    w = W.workload(2, num_requests=2, num_layers=2)
    steps = 5
    runs = [Run(w, steps), Run(w, steps)]
    twins = [Run(w, steps), Run(w, steps)]
    dev = runs[0].dev
    n_turns = w.num_layers * len(runs)
    turns = torch.zeros(2 * n_turns, dtype=torch.int32, device=dev)
    try:
        turn_step(runs, [torch.cuda.Stream(), torch.cuda.Stream()], turns, 0, w.num_layers)
        for r in twins:
            r.resolve_step(0)
        torch.cuda.synchronize()
        sel_bufs = [torch.empty_like(r.sel[0]) for r in runs]
        step = torch.ones(1, dtype=torch.int64, device=dev)
        g = torch.cuda.CUDAGraph()
        s0, s1 = torch.cuda.Stream(), torch.cuda.Stream()
        s0.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s0):
            with torch.cuda.graph(g, stream=s0):
                for r, b in zip(runs, sel_bufs):
                    b.copy_(r.sel.index_select(0, step).squeeze(0))
                step.add_(1)
                n_mb = len(runs)
                hs.hisparse_link_turns_reset(turns, n_turns, s0)
                fork = torch.cuda.Event()
                fork.record(s0)
                s1.wait_event(fork)
                for l in range(w.num_layers):
                    for i, (r, b, s) in enumerate(zip(runs, sel_bufs, (s0, s1))):
                        hs.hisparse_resolve_tables(r.cache.handle, l,
                                                   b[l * w.units:(l + 1) * w.units],
                                                   r.slots[l], r.counts[l], s)
                        ti = l * n_mb + i
                        hs.hisparse_fetch_turn(r.cache.handle, l, turns, n_turns, ti - 1, ti,
                                               256, s)
                join = torch.cuda.Event()
                join.record(s1)
                s0.wait_event(join)
        torch.cuda.synchronize()
        for t in range(1, steps):
            g.replay()
            for r in twins:
                r.resolve_step(t)
            torch.cuda.synchronize()
            scratch = torch.randn(1 << 16, device=dev).sum()  # eager work between replays
            for r, tw in zip(runs, twins):
                assert torch.equal(r.slots, tw.slots), f"slots differ at replay {t}"
                assert torch.equal(r.counts, tw.counts), f"counts differ at replay {t}"
                for l in range(w.num_layers):
                    assert (layer_cache_host(r, l) == layer_cache_host(tw, l)).all(), (t, l)
            assert (turns.view(n_turns, 2)[:, 1] == 2).all(), f"a turn unsignalled at {t}"
            del scratch
    finally:
        torch.cuda.synchronize()
        for r in runs + twins:
            r.close()
