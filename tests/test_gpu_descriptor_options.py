"""GPU parity under the descriptor's transfer options: transfer blocks of 32-256 bytes (two or
four 16-byte loads in flight per thread), fetch grids from one workgroup per unit and layer to
4096, and the three pinned host-memory kinds. Each step resolves the anchor (demand fetch),
replays its plan into one shared layer (side replay) and attends a shared layer with the replay
into the last one carried by the attention launch; slots are checked against the oracle and
every resident slot of every layer against its host record, and the shared layer's attention
output against the oracle's float64 attention over that layer's host records (max-abs 1e-2,
relative L2 5e-3)."""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, attn_desc, d2h, log
from paper_2608_07009_amd import hisparse as hs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("tb,wg,host", [
    (32, 0, hs.HISPARSE_HOST_COHERENT),
    (64, 1, hs.HISPARSE_HOST_NONCOHERENT),
    (128, 7, hs.HISPARSE_HOST_COHERENT),
    (256, 4096, hs.HISPARSE_HOST_UNCACHED),
])
def test_transfer_options_match_oracle(tb, wg, host):
    steps, NL = 6, 3
    w = W.workload(1, num_requests=3, num_layers=NL, share_group=NL)
    U, k, B, L, R = w.units, w.k, w.B, w.L, w.record_bytes
    log(f"test_transfer_options_match_oracle tb={tb} wg={wg} host={host}")
    run = Run(w, steps, transfer_block_bytes=tb, fetch_workgroups=wg, host_memory=host)
    try:
        h, dev = run.cache.handle, run.dev
        ad = attn_desc(w)
        nb = hs.hisparse_decode_workspace_bytes(U, k, R, ad)
        ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        out = torch.empty((U, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
        orc = oracle.OracleCache(U, L, B, k)
        for t in range(steps):
            hs.hisparse_resolve(h, 0, run.sel_ptr(t, 0), run.slots[0], run.counts[0], run.stream)
            hs.hisparse_prefetch_layer(h, 0, 1, run.stream)
            q_host = W.queries(w, t, 1)
            q = torch.from_numpy(q_host.view(np.int16)).to(dev)
            hs.hisparse_sparse_decode_prefetch(h, 1, q, run.slots[0], out, ad, ws, nb, 0, 2, 1,
                                               run.stream)
            torch.cuda.synchronize()
            e_slots, e_counts, _, _, bad = orc.resolve(run.sel_host[t, 0:U])
            assert bad == 0
            assert (run.slots[0].cpu().numpy() == e_slots).all(), f"slots step {t}"
            assert (run.counts[0].cpu().numpy() == e_counts).all(), f"counts step {t}"
            # the attention of the shared layer over its own records, through the anchor's slots
            o = out.cpu().numpy()
            host1 = run.cache.host_view(1)
            for u in range(U):
                ref = oracle.sparse_decode(q_host[u], host1[u].view(np.uint16).reshape(L, -1),
                                           run.sel_host[t, u], d_qk=w.d_qk, d_v=w.d_v,
                                           v_off=w.v_offset, token_elems=w.token_elems,
                                           tokens_per_record=w.tokens_per_record, scale=w.scale)
                err = float(np.abs(o[u] - ref).max())
                rl2 = float(np.linalg.norm(o[u] - ref) / np.linalg.norm(ref))
                assert err <= 1e-2 and rl2 <= 5e-3, f"attention step {t} unit {u}: {err} {rl2}"
            for l in range(NL):
                ptr, n = run.cache.layer_cache(l)
                cache = d2h(ptr, n).reshape(U, B, R)
                host_v = run.cache.host_view(l)
                for u in range(U):
                    res = np.nonzero(orc.slot_pos[u] >= 0)[0]
                    assert (cache[u][res] == host_v[u][orc.slot_pos[u][res]]).all(), \
                        f"step {t} layer {l} unit {u}"
        assert run.cache.check_errors()[0] == hs.HISPARSE_OK
    finally:
        torch.cuda.synchronize()
        run.close()
