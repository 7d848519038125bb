"""Exact layer-wise prefetch (Section 3.5) on the GPU.

Shared layers reuse their anchor's selection and slot table; the anchor's miss plan is replayed
into each shared layer's cache on a side stream. Checks:
  * equivalence: replaying the plan gives the same cache contents as resolving the shared layer
    itself with the same selection (the canonical LRU is a deterministic function of the
    selection stream);
  * every resident slot of every shared layer holds that layer's own host record;
  * shared-layer attention through the anchor's slots equals attention over the fully resident
    KV of that layer (bit-identical) and the oracle (tolerance);
  * the side-stream/event ordering: the anchor's next resolve never runs before the previous
    replays finish (checked by results, over many steps).
"""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, attn_desc, d2h, layer_cache_host, log
from paper_2608_07009_amd import HiSparseCache, hisparse as hs

pytestmark = pytest.mark.gpu


def test_replay_equals_independent_resolve():
    w = W.workload(1, num_layers=2, share_group=2)
    steps = 24
    dev = torch.device("cuda:0")
    shared = HiSparseCache.for_workload(w)
    indep = HiSparseCache.for_workload(w.__class__(**{**w.__dict__, "share_group": 1}))
    try:
        for c in (shared, indep):
            for l in range(2):
                W.fill_kv(c.host_pool(l)[0], w, l)
        sel = torch.from_numpy(W.selection_streams(w, steps=steps)).to(dev)  # [steps][1][k]
        s_a = torch.empty((1, w.k), dtype=torch.int32, device=dev)
        s_b0 = torch.empty_like(s_a)
        s_b1 = torch.empty_like(s_a)
        st = torch.cuda.current_stream()
        for t in range(steps):
            hs.hisparse_resolve(shared.handle, 0, sel[t], s_a, None, st)
            hs.hisparse_prefetch_layer(shared.handle, 0, 1, st)
            hs.hisparse_resolve(indep.handle, 0, sel[t], s_b0, None, st)
            hs.hisparse_resolve(indep.handle, 1, sel[t], s_b1, None, st)
            assert torch.equal(s_a, s_b0) and torch.equal(s_a, s_b1)
            pa, na = shared.layer_cache(1)
            pb, nb = indep.layer_cache(1)
            assert (d2h(pa, na) == d2h(pb, nb)).all(), f"step {t}"
    finally:
        shared.close()
        indep.close()


@pytest.mark.parametrize("cfg,steps", [(1, 16), (5, 6)])
def test_prefetch_side_stream(cfg, steps):
    base = W.workload(cfg)
    if cfg == 1:
        base = W.workload(1, num_layers=7, share_group=4)  # anchors 0 and 4
    run = Run(base, steps)
    w = run.w
    log(f"test_prefetch_side_stream {w.name} layers={w.num_layers} anchors={w.anchors}")
    try:
        main = torch.cuda.current_stream()
        side = torch.cuda.Stream()
        ad = attn_desc(w)
        ws = torch.empty(hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad),
                         dtype=torch.uint8, device=run.dev)
        outs = {l: torch.empty((w.units, w.q_heads, w.d_v), dtype=torch.float32,
                               device=run.dev) for l in range(w.num_layers)}
        orcs = {l: oracle.OracleCache(w.units, w.L, w.B, w.k) for l in w.anchors}
        check_layers = sorted({1, w.num_layers - 1} - set(w.anchors))
        for t in range(steps):
            q = {l: torch.from_numpy(W.queries(w, t, l).view(np.int16)).to(run.dev)
                 for l in check_layers}
            for a in w.anchors:
                hs.hisparse_resolve(run.cache.handle, a, run.sel_ptr(t, a), run.slots[a],
                                    run.counts[a], main)
                ev = torch.cuda.Event()
                ev.record(main)
                side.wait_event(ev)
                done = {}
                for s in range(a + 1, min(a + w.share_group, w.num_layers)):
                    hs.hisparse_prefetch_layer(run.cache.handle, a, s, side)
                    done[s] = torch.cuda.Event()
                    done[s].record(side)
                for s, e in done.items():
                    main.wait_event(e)
                    if s in check_layers:
                        hs.hisparse_sparse_decode(run.cache.handle, s, q[s], run.slots[a],
                                                  outs[s], ad, ws, ws.numel(), main)
            torch.cuda.synchronize()
            for a in w.anchors:
                sel = run.sel_host[t, (a // w.share_group) * w.units:
                                   (a // w.share_group + 1) * w.units]
                e_slots, _, _, _, bad = orcs[a].resolve(sel)
                assert bad == 0 and (run.slots[a].cpu().numpy() == e_slots).all()
            if t in (0, steps - 1):
                for s in check_layers:
                    a = s - s % w.share_group
                    img = layer_cache_host(run, s)
                    host = run.cache.host_view(s)
                    sp = orcs[a].slot_pos
                    for u in range(w.units):
                        res = np.nonzero(sp[u] >= 0)[0]
                        assert (img[u, res] == host[u, sp[u, res]]).all(), f"layer {s} step {t}"
                    # attention of the shared layer vs its resident KV and the oracle
                    resident = torch.from_numpy(host.reshape(-1)).to(run.dev)
                    sel_dev = run.sel[t, (a // w.share_group) * w.units:
                                      (a // w.share_group + 1) * w.units]
                    ref_dev = torch.empty_like(outs[s])
                    hs.hisparse_sparse_decode_pool(resident, w.L, w.record_bytes, w.units, w.k,
                                                   q[s], sel_dev, ref_dev, ad, ws, ws.numel(),
                                                   main)
                    torch.cuda.synchronize()
                    assert torch.equal(ref_dev, outs[s])
                    del resident
                    qh = W.queries(w, t, s)
                    sel0 = run.sel_host[t, (a // w.share_group) * w.units]
                    ref = oracle.sparse_decode(qh[0], host[0].view(np.uint16).reshape(w.L, -1),
                                               sel0, d_qk=w.d_qk, d_v=w.d_v, v_off=w.v_offset,
                                               token_elems=w.token_elems,
                                               tokens_per_record=w.tokens_per_record,
                                               scale=w.scale)
                    o = outs[s].cpu().numpy()[0]
                    assert np.abs(o - ref).max() <= 1e-2
                    assert np.linalg.norm(o - ref) / np.linalg.norm(ref) <= 5e-3
                    log(f"  step {t} shared layer {s}: ok")
    finally:
        run.close()


def test_decode_layers_batch_matches_resident():
    """One launch for an anchor and its shared layers (all reading the anchor's slots): for
    every layer, bit-identical to the same plan over the stacked, fully resident KV of those
    layers (positions instead of slots), and within the oracle's tolerance."""
    G = 4
    w = W.workload(2, num_layers=G, share_group=G, num_requests=3)
    steps = 3
    log(f"test_decode_layers_batch_matches_resident {w.name} units={w.units}")
    run = Run(w, steps)
    try:
        U, k, H = w.units, w.k, w.q_heads
        for t in range(steps):
            run.resolve_step(t, prefetch=True)
        t = steps - 1
        ad = attn_desc(w)
        q_host = np.stack([W.queries(w, t, l) for l in range(G)])       # [G][U][H][d_qk]
        q = torch.from_numpy(q_host.view(np.int16)).to(run.dev)
        ws = torch.empty(hs.hisparse_decode_workspace_bytes(G * U, k, w.record_bytes, ad),
                         dtype=torch.uint8, device=run.dev)
        out = torch.empty((G, U, H, w.d_v), dtype=torch.float32, device=run.dev)
        hs.hisparse_sparse_decode_layers(run.cache.handle, 0, G, q, run.slots[0], out, ad, ws,
                                         ws.numel(), run.stream)
        hosts = [run.cache.host_view(l) for l in range(G)]               # [U][L][R] each
        pool = torch.from_numpy(np.ascontiguousarray(np.stack(hosts)).reshape(-1)).to(run.dev)
        sel = run.sel_host[t, 0:U]                                       # anchor 0's streams
        idx = torch.from_numpy(np.ascontiguousarray(np.tile(sel, (G, 1)))).to(run.dev)
        ref = torch.empty_like(out)
        hs.hisparse_sparse_decode_pool(pool, w.L, w.record_bytes, G * U, k, q, idx, ref, ad, ws,
                                       ws.numel(), run.stream)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), "placement changed the batched output"
        o = out.cpu().numpy()
        for l, u in [(0, 0), (G - 1, U - 1), (1, 1)]:
            e = oracle.sparse_decode(q_host[l, u], hosts[l][u].view(np.uint16).reshape(w.L, -1),
                                     sel[u], d_qk=w.d_qk, d_v=w.d_v, v_off=w.v_offset,
                                     token_elems=w.token_elems,
                                     tokens_per_record=w.tokens_per_record, scale=w.scale)
            assert np.abs(o[l, u] - e).max() <= 1e-2
            assert np.linalg.norm(o[l, u] - e) / np.linalg.norm(e) <= 5e-3
        with pytest.raises(hs.HisparseError):   # spans two share groups
            hs.hisparse_sparse_decode_layers(run.cache.handle, 2, 3, q, run.slots[0], out, ad,
                                             ws, ws.numel(), run.stream)
    finally:
        run.close()


def test_fetch_group_equals_fetch_and_replays():
    """One launch for the anchor's fetch and its shared layers' replays, and the multi-layer
    replay launch on a side stream, leave every layer's cache byte-identical to hisparse_fetch
    followed by one hisparse_prefetch_layer per shared layer; bad layer ranges are argument
    errors."""
    G = 4
    w = W.workload(2, num_layers=G, share_group=G, num_requests=2)
    steps = 4
    log(f"test_fetch_group_equals_fetch_and_replays {w.name}")
    grouped = Run(w, steps)
    single = Run(w, steps)
    multi = Run(w, steps)
    side = torch.cuda.Stream()
    try:
        for t in range(steps):
            hs.hisparse_resolve_tables(grouped.cache.handle, 0, grouped.sel_ptr(t, 0),
                                       grouped.slots[0], grouped.counts[0], grouped.stream)
            hs.hisparse_fetch_group(grouped.cache.handle, 0, G, grouped.stream)
            single.resolve_step(t, prefetch=True)
            # the replays on a side stream, started right after the resolve, as two launches
            hs.hisparse_resolve_tables(multi.cache.handle, 0, multi.sel_ptr(t, 0),
                                       multi.slots[0], multi.counts[0], multi.stream)
            resolved = torch.cuda.Event()
            resolved.record(multi.stream)
            side.wait_event(resolved)
            hs.hisparse_prefetch_layers(multi.cache.handle, 0, 1, 2, side)
            hs.hisparse_prefetch_layers(multi.cache.handle, 0, 3, 1, side)
            hs.hisparse_fetch(multi.cache.handle, 0, multi.stream)
            replayed = torch.cuda.Event()
            replayed.record(side)
            multi.stream.wait_event(replayed)  # before the anchor's next resolve
        torch.cuda.synchronize()
        assert torch.equal(grouped.slots[0], single.slots[0])
        assert torch.equal(multi.slots[0], single.slots[0])
        for l in range(G):
            ref = layer_cache_host(single, l)
            assert (layer_cache_host(grouped, l) == ref).all(), f"group fetch, layer {l}"
            assert (layer_cache_host(multi, l) == ref).all(), f"multi-layer replay, layer {l}"
        for n in (0, G + 1):
            with pytest.raises(hs.HisparseError):
                hs.hisparse_fetch_group(grouped.cache.handle, 0, n, grouped.stream)
        with pytest.raises(hs.HisparseError):   # not an anchor layer
            hs.hisparse_fetch_group(grouped.cache.handle, 1, 2, grouped.stream)
        for first, n in ((0, 1), (1, 0), (1, G), (2, G - 1), (4, 1)):
            with pytest.raises(hs.HisparseError):
                hs.hisparse_prefetch_layers(multi.cache.handle, 0, first, n, multi.stream)
    finally:
        torch.cuda.synchronize()
        grouped.close()
        single.close()
        multi.close()


@pytest.mark.parametrize("cfg,fetch", [(2, hs.HISPARSE_FETCH_ZERO_COPY),
                                       (3, hs.HISPARSE_FETCH_ZERO_COPY),
                                       (2, hs.HISPARSE_FETCH_SDMA),
                                       (3, hs.HISPARSE_FETCH_STAGED)])
def test_decode_prefetch_equals_separate(cfg, fetch):
    """Attention of one layer carrying the replay into later shared layers in the same launch
    gives bit-identical attention outputs and byte-identical caches to the replay and the
    attention issued apart, for the latent (MLA) and the grouped-query kernels, and with the
    copy-engine path (where the replay is issued on its own first); replay ranges that include
    the attended layer, or that hisparse_prefetch_layers would refuse, are argument errors."""
    G = 4
    if cfg == 2:
        w = W.workload(2, num_layers=G, share_group=G, num_requests=2)
    else:
        w = W.workload(3, num_layers=G, share_group=G, num_requests=2)
    steps = 3
    log(f"test_decode_prefetch_equals_separate {w.name} fetch={fetch}")
    fused, apart = Run(w, steps, fetch=fetch), Run(w, steps, fetch=fetch)
    dev = fused.dev
    ad = attn_desc(w)
    nb = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad)
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    out_f = torch.empty((G, w.units, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
    out_a = torch.empty_like(out_f)
    try:
        for t in range(steps):
            q = [torch.from_numpy(W.queries(w, t, l).view(np.int16)).to(dev) for l in range(G)]
            for r in (fused, apart):
                hs.hisparse_resolve(r.cache.handle, 0, r.sel_ptr(t, 0), r.slots[0], r.counts[0],
                                    r.stream)
            h = fused.cache.handle
            hs.hisparse_sparse_decode_prefetch(h, 0, q[0], fused.slots[0], out_f[0], ad, ws, nb,
                                               0, 1, 1, fused.stream)
            hs.hisparse_sparse_decode_prefetch(h, 1, q[1], fused.slots[0], out_f[1], ad, ws, nb,
                                               0, 2, 2, fused.stream)
            for l in (2, 3):
                hs.hisparse_sparse_decode(h, l, q[l], fused.slots[0], out_f[l], ad, ws, nb,
                                          fused.stream)
            hs.hisparse_prefetch_layers(apart.cache.handle, 0, 1, G - 1, apart.stream)
            for l in range(G):
                hs.hisparse_sparse_decode(apart.cache.handle, l, q[l], apart.slots[0], out_a[l],
                                          ad, ws, nb, apart.stream)
            torch.cuda.synchronize()
            assert torch.equal(out_f, out_a), f"step {t}"
            for l in range(G):
                assert (layer_cache_host(fused, l) == layer_cache_host(apart, l)).all(), \
                    f"step {t} layer {l}"
        h = fused.cache.handle
        for layer, first, n in ((1, 1, 1), (2, 1, 3), (0, 0, 1), (0, 1, 0), (0, 2, 3), (1, 2, 9)):
            with pytest.raises(hs.HisparseError):
                hs.hisparse_sparse_decode_prefetch(h, layer, q[0], fused.slots[0], out_f[0], ad,
                                                   ws, nb, 0, first, n, fused.stream)
        with pytest.raises(hs.HisparseError):  # the replay's anchor must be an anchor layer
            hs.hisparse_sparse_decode_prefetch(h, 0, q[0], fused.slots[0], out_f[0], ad, ws, nb,
                                               1, 2, 1, fused.stream)
    finally:
        torch.cuda.synchronize()
        fused.close()
        apart.close()


@pytest.mark.parametrize("cfg", [2, 3])
def test_deferred_merge_equals_fused(cfg):
    """HISPARSE_ATTN_DEFER_MERGE + hisparse_attention_merge gives bit-identical outputs to the
    fused call for one layer, a replay-carrying layer and a batched group of layers, for the
    latent (MLA) and the grouped-query kernels."""
    G = 4
    w = W.workload(cfg, num_layers=G, share_group=G, num_requests=2)
    log(f"test_deferred_merge_equals_fused {w.name}")
    run = Run(w, 2)
    try:
        U, k, H, R, dev = w.units, w.k, w.q_heads, w.record_bytes, run.dev
        h = run.cache.handle
        hs.hisparse_resolve(h, 0, run.sel_ptr(0, 0), run.slots[0], run.counts[0], run.stream)
        ad = attn_desc(w)
        adf = attn_desc(w)
        adf.flags = hs.HISPARSE_ATTN_DEFER_MERGE
        nb = max(hs.hisparse_decode_workspace_bytes(n, k, R, ad) for n in (U, G * U))
        ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        q = torch.from_numpy(np.stack([W.queries(w, 0, l) for l in range(G)]).view(np.int16)).to(dev)
        fused = torch.empty((G, U, H, w.d_v), dtype=torch.float32, device=dev)
        deferred = torch.full_like(fused, float("nan"))
        # one layer
        hs.hisparse_sparse_decode(h, 0, q[0], run.slots[0], fused[0], ad, ws, nb, run.stream)
        hs.hisparse_sparse_decode(h, 0, q[0], run.slots[0], deferred[0], adf, ws, nb, run.stream)
        torch.cuda.synchronize()
        assert torch.isnan(deferred[0]).all()  # the deferred call leaves the output alone
        hs.hisparse_attention_merge(U, k, R, adf, deferred[0], ws, nb, run.stream)
        # attention of layer 0 carrying the replay into layers 1..3 (idempotent: same plan)
        hs.hisparse_sparse_decode_prefetch(h, 0, q[0], run.slots[0], fused[1], ad, ws, nb, 0, 1,
                                           G - 1, run.stream)
        hs.hisparse_sparse_decode_prefetch(h, 0, q[0], run.slots[0], deferred[1], adf, ws, nb, 0,
                                           1, G - 1, run.stream)
        hs.hisparse_attention_merge(U, k, R, adf, deferred[1], ws, nb, run.stream)
        torch.cuda.synchronize()
        assert torch.equal(fused[:2], deferred[:2])
        assert torch.equal(fused[0], fused[1])
        # the whole group in one launch: units = G * U
        f_all, d_all = torch.empty_like(fused), torch.full_like(fused, float("nan"))
        hs.hisparse_sparse_decode_layers(h, 0, G, q, run.slots[0], f_all, ad, ws, nb, run.stream)
        hs.hisparse_sparse_decode_layers(h, 0, G, q, run.slots[0], d_all, adf, ws, nb, run.stream)
        hs.hisparse_attention_merge(G * U, k, R, adf, d_all, ws, nb, run.stream)
        torch.cuda.synchronize()
        assert torch.equal(f_all, d_all)  # (its split plan is that of G * U units)
        with pytest.raises(hs.HisparseError):  # workspace smaller than the plan needs
            hs.hisparse_attention_merge(G * U, k, R, adf, d_all, ws, 256, run.stream)
    finally:
        torch.cuda.synchronize()
        run.close()


@pytest.mark.parametrize("cfg,fetch,share", [(2, hs.HISPARSE_FETCH_ZERO_COPY, 64),
                                             (2, hs.HISPARSE_FETCH_ZERO_COPY, 1),
                                             (2, hs.HISPARSE_FETCH_ZERO_COPY, 256),
                                             (3, hs.HISPARSE_FETCH_ZERO_COPY, 200),
                                             (2, hs.HISPARSE_FETCH_SDMA, 64),
                                             (2, hs.HISPARSE_FETCH_STAGED, 100)])
def test_merge_carried_replay_equals_separate(cfg, fetch, share):
    """The overlap schedule with the merges starting the replay into the layer after next
    (hisparse_attention_merge_prefetch over the first share/256 of each unit's plan) and the
    following attention carrying the rest (hisparse_sparse_decode_prefetch_part): attention
    outputs bit-identical and caches byte-identical to the replay and the attention issued apart,
    every planned record copied once; bad plan ranges are argument errors."""
    G = 4
    w = W.workload(cfg, num_layers=G, share_group=G, num_requests=2)
    steps = 3
    log(f"test_merge_carried_replay_equals_separate {w.name} fetch={fetch} share={share}")
    split, apart = Run(w, steps, fetch=fetch), Run(w, steps, fetch=fetch)
    dev = split.dev
    ad = attn_desc(w)
    adf = attn_desc(w)
    adf.flags = hs.HISPARSE_ATTN_DEFER_MERGE
    nb = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad)
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    out_s = torch.empty((G, w.units, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
    out_a = torch.empty_like(out_s)
    try:
        for t in range(steps):
            q = [torch.from_numpy(W.queries(w, t, l).view(np.int16)).to(dev) for l in range(G)]
            for r in (split, apart):
                hs.hisparse_resolve(r.cache.handle, 0, r.sel_ptr(t, 0), r.slots[0], r.counts[0],
                                    r.stream)
            h, st = split.cache.handle, split.stream
            for l in range(G - 1):
                lo = share if l >= 1 else 0
                hs.hisparse_sparse_decode_prefetch_part(h, l, q[l], split.slots[0], out_s[l], adf,
                                                        ws, nb, 0, l + 1, 1, lo, 256, st)
                if l + 2 < G:
                    hs.hisparse_attention_merge_prefetch(h, adf, out_s[l], ws, nb, 0, l + 2, 1, 0,
                                                         share, st)
                else:
                    hs.hisparse_attention_merge(w.units, w.k, w.record_bytes, adf, out_s[l], ws,
                                                nb, st)
            hs.hisparse_sparse_decode(h, G - 1, q[G - 1], split.slots[0], out_s[G - 1], ad, ws,
                                      nb, st)
            hs.hisparse_prefetch_layers(apart.cache.handle, 0, 1, G - 1, apart.stream)
            for l in range(G):
                hs.hisparse_sparse_decode(apart.cache.handle, l, q[l], apart.slots[0], out_a[l],
                                          ad, ws, nb, apart.stream)
            torch.cuda.synchronize()
            assert torch.equal(out_s, out_a), f"step {t}"
            for l in range(G):
                assert (layer_cache_host(split, l) == layer_cache_host(apart, l)).all(), \
                    f"step {t} layer {l}"
        h, st = split.cache.handle, split.stream
        for lo, hi in ((-1, 10), (10, 9), (0, 257)):
            with pytest.raises(hs.HisparseError):
                hs.hisparse_attention_merge_prefetch(h, adf, out_s[0], ws, nb, 0, 2, 1, lo, hi, st)
            with pytest.raises(hs.HisparseError):
                hs.hisparse_sparse_decode_prefetch_part(h, 0, q[0], split.slots[0], out_s[0], adf,
                                                        ws, nb, 0, 1, 1, lo, hi, st)
        with pytest.raises(hs.HisparseError):  # a replay target outside the anchor's group
            hs.hisparse_attention_merge_prefetch(h, adf, out_s[0], ws, nb, 0, 4, 1, 0, 64, st)
    finally:
        torch.cuda.synchronize()
        split.close()
        apart.close()


@pytest.mark.parametrize("requests", [1, 2])
def test_carries_replay_hint_equals_separate(requests):
    """The overlap schedule with HISPARSE_ATTN_CARRIES_REPLAY on the replay-carrying attention
    calls and on their merges, the last layer's attention without it (one or two requests of 128
    latent heads, k = 2048: one token group per workgroup, where the hint halves the splits):
    outputs bit-identical to the same plans' attention issued apart from the replay, caches
    byte-identical."""
    G = 4
    w = W.workload(2, num_layers=G, share_group=G, num_requests=requests)
    steps = 2
    log(f"test_carries_replay_hint_equals_separate {w.name} units={w.units}")
    split, apart = Run(w, steps), Run(w, steps)
    dev = split.dev
    ad = attn_desc(w)
    adc = attn_desc(w, 0, hs.HISPARSE_ATTN_CARRIES_REPLAY)
    adcf = attn_desc(w, 0, hs.HISPARSE_ATTN_CARRIES_REPLAY | hs.HISPARSE_ATTN_DEFER_MERGE)
    nb = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad)
    nbc = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, adc)
    assert 0 < nbc < nb  # fewer split partials
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    out_s = torch.empty((G, w.units, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
    out_a = torch.empty_like(out_s)
    try:
        for t in range(steps):
            q = [torch.from_numpy(W.queries(w, t, l).view(np.int16)).to(dev) for l in range(G)]
            for r in (split, apart):
                hs.hisparse_resolve(r.cache.handle, 0, r.sel_ptr(t, 0), r.slots[0], r.counts[0],
                                    r.stream)
            h, st = split.cache.handle, split.stream
            for l in range(G - 1):
                hs.hisparse_sparse_decode_prefetch(h, l, q[l], split.slots[0], out_s[l], adcf, ws,
                                                   nbc, 0, l + 1, 1, st)
                hs.hisparse_attention_merge(w.units, w.k, w.record_bytes, adcf, out_s[l], ws, nbc,
                                            st)
            hs.hisparse_sparse_decode(h, G - 1, q[G - 1], split.slots[0], out_s[G - 1], ad, ws, nb,
                                      st)
            hs.hisparse_prefetch_layers(apart.cache.handle, 0, 1, G - 1, apart.stream)
            for l in range(G):
                hs.hisparse_sparse_decode(apart.cache.handle, l, q[l], apart.slots[0], out_a[l],
                                          adc if l < G - 1 else ad, ws, nb, apart.stream)
            torch.cuda.synchronize()
            assert torch.equal(out_s, out_a), f"step {t}"
            for l in range(G):
                assert (layer_cache_host(split, l) == layer_cache_host(apart, l)).all(), \
                    f"step {t} layer {l}"
    finally:
        torch.cuda.synchronize()
        split.close()
        apart.close()
