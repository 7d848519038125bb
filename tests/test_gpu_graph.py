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
from hs_harness import Run, attn_desc, log
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
