"""GPU parity of the write-through of generated records (Section 3.3 (4)).

A decode loop over a growing context: every step resolves the anchor's selection (whose window
follows the newest records), fetches its misses, replays them into the shared layer, then
appends each unit's newly generated record to both layers. Checked against the oracle, in which
an admission is a one-entry resolve event:
  * the admission slot of every unit and step, and the step's slots and counts, bit-exact;
  * the final slot map, stamps, clock and page table, bit-exact;
  * every resident slot of both layers holds that layer's record of the slot's position
    (prefill records from the host pool, appended records as generated);
  * the host pools hold every appended record after the write-through, and an appended record
    that was evicted and selected again comes back from the host pool intact.
"""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, d2h, log
from paper_2608_07009_amd import hisparse as hs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fetch", [hs.HISPARSE_FETCH_ZERO_COPY, hs.HISPARSE_FETCH_SDMA])
def test_append_write_through_matches_oracle(fetch):
    steps = 60
    base = W.workload(1, num_layers=2, share_group=2, num_requests=2)
    L0 = base.L
    w = W.workload(1, num_layers=2, share_group=2, num_requests=2, L=L0 + steps)
    U, k, B, R = w.units, w.k, w.B, w.record_bytes
    log(f"test_append_write_through_matches_oracle fetch={fetch} units={U} steps={steps}")
    run = Run(w, steps, fill=False, fetch=fetch)
    try:
        dev = run.dev
        for l in range(2):
            host = run.cache.host_view(l)
            host[:] = 0xAB  # appended positions must come from the write-through
            ptr = run.cache.host_pool(l)[0]
            for u in range(U):  # prefill [0, L0) of every unit (the pool holds L0 + steps)
                W.fill_kv(ptr + u * w.L * R, base, l, u, 1)
        sel = W.grow_streams(base, W.selection_streams(base, steps=steps))  # [steps][U][k]
        # from step 52 on, one entry per unit is replaced by the record appended 50 steps
        # earlier: out of the window for 17 steps and evicted, it must come back from the host
        back = 50
        for t in range(52, steps):
            sel[t, :, 0] = L0 + (t - back)
        sel_d = torch.from_numpy(sel).to(dev)
        new = np.stack([np.stack([np.stack([W.kv_records(base, l, u, [L0 + t])[0]
                                            for u in range(U)]) for l in range(2)])
                        for t in range(steps)])  # uint16 [steps][layers][U][R/2]
        new_d = torch.from_numpy(new.view(np.int16)).to(dev)
        pos_d = torch.empty(U, dtype=torch.int32, device=dev)
        aslots = torch.empty(U, dtype=torch.int32, device=dev)
        orc = oracle.OracleCache(U, w.L, B, k)
        for t in range(steps):
            hs.hisparse_resolve(run.cache.handle, 0, sel_d[t], run.slots[0], run.counts[0],
                                run.stream)
            hs.hisparse_prefetch_layer(run.cache.handle, 0, 1, run.stream)
            pos_d.fill_(L0 + t)
            hs.hisparse_append(run.cache.handle, 0, 2, pos_d, new_d[t], aslots, run.stream)
            torch.cuda.synchronize()
            e_slots, e_counts, e_pp, _, bad = orc.resolve(sel[t])
            assert bad == 0
            assert (run.slots[0].cpu().numpy() == e_slots).all(), f"slots at step {t}"
            assert (run.counts[0].cpu().numpy() == e_counts).all(), f"counts at step {t}"
            e_adm = [orc.admit_unit(u, L0 + t) for u in range(U)]
            assert all(rc == oracle.OK for rc, _, _ in e_adm)
            assert aslots.cpu().numpy().tolist() == [s for _, s, _ in e_adm], f"admission {t}"
            if t >= 52:  # the re-selected old record was a miss, fetched from the host pool
                for u in range(U):
                    assert L0 + t - back in e_pp[u].tolist()
                    s0 = int(e_slots[u, 0])
                    for l in range(2):
                        ptr, _ = run.cache.layer_cache(l)
                        got = d2h(ptr + (u * B + s0) * R, R).view(np.uint16)
                        assert (got == new[t - back, l, u]).all(), f"refetch {t} {l} {u}"
        assert run.cache.check_errors()[0] == hs.HISPARSE_OK
        st = run.cache.read_state(0)
        assert (st["slot_pos"] == orc.slot_pos).all()
        assert (st["slot_ts"] == orc.slot_ts).all()
        assert (st["clock"] == orc.clock).all()
        assert (st["page_table"] == orc.pt).all()
        # cache contents: every resident slot of both layers holds its position's record
        for l in range(2):
            ptr, n = run.cache.layer_cache(l)
            cache = d2h(ptr, n).reshape(U, B, R)
            host = run.cache.host_view(l)
            for u in range(U):
                res = np.nonzero(orc.slot_pos[u] >= 0)[0]
                expect = host[u][orc.slot_pos[u][res]]
                assert (cache[u][res] == expect).all(), f"layer {l} unit {u}"
                appended = host[u][L0:L0 + steps].view(np.uint16)
                assert (appended == new[:, l, u]).all(), f"write-through, layer {l} unit {u}"
    finally:
        torch.cuda.synchronize()
        run.close()


def test_append_argument_errors():
    w = W.workload(1, num_layers=3, share_group=2, num_requests=1)
    run = Run(w, 1, fill=False)
    try:
        dev = run.dev
        pos = torch.zeros(1, dtype=torch.int32, device=dev)
        rec = torch.zeros((2, 1, w.record_bytes // 2), dtype=torch.int16, device=dev)
        slots = torch.empty(1, dtype=torch.int32, device=dev)
        h = run.cache.handle
        for anchor, n in ((1, 1), (0, 0), (0, 3), (2, 2)):  # not an anchor / group sizes
            with pytest.raises(hs.HisparseError):
                hs.hisparse_append(h, anchor, n, pos, rec, slots, run.stream)
        # a position outside [0, L) is latched as a bad selection; the slot reads -1
        pos.fill_(w.L)
        hs.hisparse_append(h, 0, 2, pos, rec, slots, run.stream)
        torch.cuda.synchronize()
        assert slots.item() == -1
        assert run.cache.check_errors()[0] == hs.HISPARSE_ERR_BAD_SELECTION
    finally:
        torch.cuda.synchronize()
        run.close()
