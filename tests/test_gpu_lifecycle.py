"""GPU parity of the request lifecycle (Section 3.3 (1) prefill and staging, (2) admission).

Every request's prefill records are staged from device memory into the host pools by the copy
engines (hisparse_stage); the decode loop then resolves and fetches them. Midway, one request
finishes: its slot is released (its units go back to the cold state) and a new request with
different records and selections is admitted into it and staged, in two partial ranges. Checked
against the oracle, in which the admission resets the unit:
  * host pools equal the staged device bytes, bit-exact;
  * slots and counts of every unit and step, bit-exact, and the final tables;
  * every resident slot holds the record of its position from the current request's pool;
  * the other requests' units are unaffected by the release.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, d2h, expected_order, log
from paper_2608_07009_amd import hisparse as hs

pytestmark = pytest.mark.gpu


def device_records(w, layers, unit0, n_units, rec0, n_rec):
    """Device tensor [layers][n_units][n_rec][R] of w's records (its seed) for staging."""
    R = w.record_bytes
    host = np.empty((len(layers), n_units, n_rec, R), dtype=np.uint8)
    for j, l in enumerate(layers):
        W.fill_kv(host[j].ctypes.data, w, l, unit0, n_units, rec0, n_rec)
    return host, torch.from_numpy(host).to("cuda:0")


@pytest.mark.parametrize("cfg,requests", [(1, 3), (3, 2)])
def test_release_admit_stage_matches_oracle(cfg, requests):
    steps, swap, NL = 24, 10, 2
    w = W.workload(cfg, num_layers=NL, share_group=NL, num_requests=requests)
    w_new = dataclasses.replace(w, seed=w.seed + 7)  # the request admitted midway
    U, H, k, B, L, R = w.units, w.units_per_request, w.k, w.B, w.L, w.record_bytes
    log(f"test_release_admit_stage_matches_oracle cfg={cfg} units={U} H={H} k={k} B={B} L={L}")
    run = Run(w, steps, fill=False)
    try:
        h = run.cache.handle
        for l in range(NL):
            run.cache.host_view(l)[:] = 0xCD
        got = [hs.hisparse_request_acquire(h) for _ in range(requests)]
        assert got == list(range(requests))
        with pytest.raises(hs.HisparseError) as e:
            hs.hisparse_request_acquire(h)
        assert e.value.status == hs.HISPARSE_ERR_FULL
        # prefill staging of every request, all layers in one call
        src_h, src_d = device_records(w, range(NL), 0, U, 0, L)
        hs.hisparse_stage(h, 0, NL, 0, U, 0, L, src_d, src_d[0].numel(), run.stream)
        torch.cuda.synchronize()
        for l in range(NL):
            assert (run.cache.host_view(l).reshape(U, L, R) == src_h[l]).all(), f"staged {l}"
        sel_old = run.sel_host
        sel_new = W.selection_streams(w_new, steps=steps)
        r = requests - 1  # the request that finishes at `swap`
        mine = slice(r * H, (r + 1) * H)
        orc = oracle.OracleCache(U, L, B, k)
        for t in range(steps):
            if t == swap:
                hs.hisparse_request_release(h, r, run.stream)
                with pytest.raises(hs.HisparseError):  # not taken any more
                    hs.hisparse_request_release(h, r, run.stream)
                assert hs.hisparse_request_acquire(h) == r
                half = L // 2
                new_h1, new_d1 = device_records(w_new, range(NL), r * H, H, 0, half)
                new_h2, new_d2 = device_records(w_new, range(NL), r * H, H, half, L - half)
                hs.hisparse_stage(h, 0, NL, r * H, H, 0, half, new_d1, new_d1[0].numel(),
                                  run.stream)
                for l in range(NL):  # one layer per call for the second range
                    hs.hisparse_stage(h, l, 1, r * H, H, half, L - half, new_d2[l], 0,
                                      run.stream)
                torch.cuda.synchronize()
                for l in range(NL):
                    pool = run.cache.host_view(l).reshape(U, L, R)
                    assert (pool[mine, :half] == new_h1[l]).all(), f"staged new {l}"
                    assert (pool[mine, half:] == new_h2[l]).all(), f"staged new {l}"
                    assert (pool[:r * H] == src_h[l][:r * H]).all(), f"others {l}"
                for u in range(r * H, (r + 1) * H):
                    orc.reset_unit(u)
                st = run.cache.read_state(0)
                assert (st["clock"][mine] == 0).all() and (st["slot_pos"][mine] == -1).all()
                assert (st["page_table"][mine] == -1).all()
                assert (st["order"][mine] == np.arange(B)).all()
            sel = sel_old[t].copy()
            if t >= swap:
                sel[mine] = sel_new[t - swap][mine]
            sel_d = torch.from_numpy(sel).to(run.dev)
            hs.hisparse_resolve(h, 0, sel_d, run.slots[0], run.counts[0], run.stream)
            hs.hisparse_prefetch_layer(h, 0, 1, run.stream)
            torch.cuda.synchronize()
            e_slots, e_counts, _, _, bad = orc.resolve(sel)
            assert bad == 0
            assert (run.slots[0].cpu().numpy() == e_slots).all(), f"slots step {t}"
            assert (run.counts[0].cpu().numpy() == e_counts).all(), f"counts step {t}"
        assert run.cache.check_errors()[0] == hs.HISPARSE_OK
        st = run.cache.read_state(0)
        assert (st["slot_pos"] == orc.slot_pos).all()
        assert (st["slot_ts"] == orc.slot_ts).all()
        assert (st["clock"] == orc.clock).all()
        assert (st["page_table"] == orc.pt).all()
        assert (st["order"] == expected_order(orc.slot_ts)).all()
        for l in range(NL):
            ptr, n = run.cache.layer_cache(l)
            cache = d2h(ptr, n).reshape(U, B, R)
            pool = run.cache.host_view(l).reshape(U, L, R)
            for u in range(U):
                res = np.nonzero(orc.slot_pos[u] >= 0)[0]
                assert (cache[u][res] == pool[u][orc.slot_pos[u][res]]).all(), f"layer {l} {u}"
    finally:
        torch.cuda.synchronize()
        run.close()


def test_lifecycle_argument_errors():
    w = W.workload(1, num_layers=2, share_group=1, num_requests=2)
    run = Run(w, 1, fill=False)
    try:
        h = run.cache.handle
        U, L, R = w.units, w.L, w.record_bytes
        src = torch.zeros((2, U, 4, R), dtype=torch.uint8, device=run.dev)
        bad_reset = ((-1, 1), (0, 0), (1, 2), (U, 1))
        for fu, nu in bad_reset:
            with pytest.raises(hs.HisparseError):
                hs.hisparse_reset_units(h, fu, nu, run.stream)
        bad_stage = (  # (first_layer, num_layers, first_unit, num_units, rec0, n_rec, stride)
            (-1, 1, 0, 1, 0, 4, 0), (1, 2, 0, 1, 0, 4, 0), (0, 1, 0, U + 1, 0, 4, 0),
            (0, 1, 0, 1, -1, 4, 0), (0, 1, 0, 1, L - 3, 4, 0), (0, 1, 0, 1, 0, 0, 0),
            (0, 2, 0, U, 0, 4, U * 4 * R - 16))
        for fl, nl, fu, nu, r0, nr, stride in bad_stage:
            with pytest.raises(hs.HisparseError):
                hs.hisparse_stage(h, fl, nl, fu, nu, r0, nr, src, stride, run.stream)
        for req in (-1, 2, 0):  # out of range, out of range, not taken
            with pytest.raises(hs.HisparseError):
                hs.hisparse_request_release(h, req, run.stream)
        # the last records of the last unit: the upper bounds are inclusive
        hs.hisparse_stage(h, 0, 2, U - 1, 1, L - 4, 4, src, src[0].numel(), run.stream)
        hs.hisparse_reset_units(h, U - 1, 1, run.stream)
        torch.cuda.synchronize()
        assert run.cache.check_errors()[0] == hs.HISPARSE_OK
    finally:
        torch.cuda.synchronize()
        run.close()
