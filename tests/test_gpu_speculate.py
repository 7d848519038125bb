"""GPU parity of speculative cross-layer prefetch (Section 3.5, the speculative alternative).

Layers do not share selections (share group 1); every layer's selection of a step is given to
the next layer as a hint before that layer resolves. In the oracle a hint is one access event
of the target layer's canonical LRU, exactly a resolve of the hint. Checked, for the
zero-copy and copy-engine fetch paths:
  * slots and counts of every real resolve, and the hint counts {already resident, fetched},
    bit-exact at every step;
  * the final tables of every layer, bit-exact;
  * every resident slot of every layer holds its position's record (hinted records included).
"""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, expected_order, layer_cache_host, log
from paper_2608_07009_amd import hisparse as hs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fetch", [hs.HISPARSE_FETCH_ZERO_COPY, hs.HISPARSE_FETCH_SDMA,
                                   hs.HISPARSE_FETCH_STAGED])
def test_speculate_matches_oracle(fetch):
    steps, NL = 12, 3
    w = W.workload(2, num_requests=4, num_layers=NL, share_group=1)
    U, k, B, L = w.units, w.k, w.B, w.L
    log(f"test_speculate_matches_oracle fetch={fetch} units={U} layers={NL} steps={steps}")
    run = Run(w, steps, fetch=fetch)
    try:
        h = run.cache.handle
        sel = W.correlate_layers(w, run.sel_host, 0.5, seed=3)  # [steps][NL * U][k]
        sel_d = torch.from_numpy(sel).to(run.dev)
        spec_counts = torch.empty((U, 2), dtype=torch.int32, device=run.dev)
        orc = [oracle.OracleCache(U, L, B, k) for _ in range(NL)]
        for t in range(steps):
            for l in range(NL):
                s_l = sel_d[t, l * U:(l + 1) * U]
                hs.hisparse_resolve(h, l, s_l, run.slots[l], run.counts[l], run.stream)
                if l + 1 < NL:
                    hs.hisparse_speculate(h, l + 1, s_l, spec_counts, run.stream)
                torch.cuda.synchronize()
                e_slots, e_counts, _, _, bad = orc[l].resolve(sel[t, l * U:(l + 1) * U])
                assert bad == 0
                assert (run.slots[l].cpu().numpy() == e_slots).all(), f"slots {t} {l}"
                assert (run.counts[l].cpu().numpy() == e_counts).all(), f"counts {t} {l}"
                if l + 1 < NL:  # the hint: one access event of the next layer's LRU
                    _, h_counts, _, _, bad = orc[l + 1].resolve(sel[t, l * U:(l + 1) * U])
                    assert bad == 0
                    assert (spec_counts.cpu().numpy() == h_counts).all(), f"hint {t} {l + 1}"
        assert run.cache.check_errors()[0] == hs.HISPARSE_OK
        for l in range(NL):
            st = run.cache.read_state(l)
            assert (st["slot_pos"] == orc[l].slot_pos).all()
            assert (st["slot_ts"] == orc[l].slot_ts).all()
            assert (st["clock"] == orc[l].clock).all()
            assert (st["page_table"] == orc[l].pt).all()
            assert (st["order"] == expected_order(orc[l].slot_ts)).all()
            cache = layer_cache_host(run, l)
            pool = run.cache.host_view(l)
            for u in range(U):
                res = np.nonzero(orc[l].slot_pos[u] >= 0)[0]
                assert (cache[u][res] == pool[u][orc[l].slot_pos[u][res]]).all(), f"{l} {u}"
    finally:
        torch.cuda.synchronize()
        run.close()


def test_speculate_argument_errors():
    w = W.workload(1, num_layers=2, share_group=2, num_requests=1)
    run = Run(w, 1, fill=False)
    try:
        h = run.cache.handle
        hint = torch.zeros((w.units, w.k), dtype=torch.int32, device=run.dev)
        for layer in (1, -1, 2):  # shared layer, out of range
            with pytest.raises(hs.HisparseError):
                hs.hisparse_speculate(h, layer, hint, None, run.stream)
        with pytest.raises(hs.HisparseError):
            hs.hisparse_speculate(h, 0, None, None, run.stream)
        hint.fill_(w.L)  # out of range: latched, state untouched
        hs.hisparse_speculate(h, 0, hint, None, run.stream)
        torch.cuda.synchronize()
        assert run.cache.check_errors()[0] == hs.HISPARSE_ERR_BAD_SELECTION
        assert (run.cache.read_state(0)["clock"] == 0).all()
    finally:
        torch.cuda.synchronize()
        run.close()
