"""The allocation-free attention entry point (hisparse_sparse_decode_noalloc) against the same
attention with a caller workspace (hisparse_sparse_decode): identical bits on consecutive calls
that share the library's per-GPU scratch, the second smaller than the first (and a third of the
other attention kind), the float64 oracle's tolerance, and the host-side refusals."""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import Run, attn_desc, log
from paper_2608_07009_amd import hisparse as hs

pytestmark = pytest.mark.gpu


def decode_both(run, step, layer=0):
    """Resolve `step`, then the layer's attention through both entry points."""
    w, dev = run.w, run.dev
    run.resolve_step(step)
    q_host = W.queries(w, step, layer)
    q = torch.from_numpy(q_host.view(np.int16)).to(dev)
    ad = attn_desc(w)
    out_na = torch.full((w.units, w.q_heads, w.d_v), float("nan"), dtype=torch.float32,
                        device=dev)
    hs.hisparse_sparse_decode_noalloc(run.cache.handle, layer, q, run.slots[layer], out_na, ad,
                                      run.stream)
    nb = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad)
    assert 0 < nb <= hs.HISPARSE_NOALLOC_SCRATCH_BYTES
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    out_ws = torch.empty_like(out_na)
    hs.hisparse_sparse_decode(run.cache.handle, layer, q, run.slots[layer], out_ws, ad, ws, nb,
                              run.stream)
    torch.cuda.synchronize()
    return q_host, out_na.cpu().numpy(), out_ws.cpu().numpy()


def test_noalloc_matches_workspace_decode_on_consecutive_calls():
    cases = [  # the second call smaller than the first, then grouped-query attention
        W.workload(1, num_requests=6, q_heads=128),
        W.workload(1, num_requests=2, q_heads=32),
        W.workload(3, num_requests=1, num_layers=1),
    ]
    for ci, w in enumerate(cases):
        log(f"noalloc case {ci}: {w.name} units={w.units} heads={w.q_heads} k={w.k}")
        run = Run(w, steps=3)
        try:
            for t in range(3):
                q_host, o_na, o_ws = decode_both(run, t)
                assert not np.isnan(o_na).any(), f"case {ci} step {t}: output not written"
                assert o_na.tobytes() == o_ws.tobytes(), f"case {ci} step {t}"
            host = run.cache.host_view(0)
            sel = run.sel_host[2]
            for u in range(w.units):
                ref = oracle.sparse_decode(q_host[u], host[u].view(np.uint16).reshape(w.L, -1),
                                           sel[u], d_qk=w.d_qk, d_v=w.d_v, v_off=w.v_offset,
                                           token_elems=w.token_elems,
                                           tokens_per_record=w.tokens_per_record, scale=w.scale)
                err = float(np.abs(o_na[u] - ref).max())
                rl2 = float(np.linalg.norm(o_na[u] - ref) / np.linalg.norm(ref))
                assert err <= 1e-2 and rl2 <= 5e-3, (ci, u, err, rl2)
            assert run.cache.check_errors()[0] == hs.HISPARSE_OK
        finally:
            torch.cuda.synchronize()
            run.close()


def test_noalloc_refuses_oversize_and_deferred_calls():
    w = W.workload(2, num_requests=8, num_layers=1)
    run = Run(w, steps=1)
    try:
        dev = run.dev
        run.resolve_step(0)
        # 256 heads in as many splits as the plan allows (at least 16 of 2048 tokens): 8 units x
        # >= 16 x 256 x 2 KiB of partials > 64 MiB
        big = hs.AttnDesc(256, 576, 512, 0, 1, 64, w.scale, 0)
        assert hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, big) > \
            hs.HISPARSE_NOALLOC_SCRATCH_BYTES
        q = torch.zeros((w.units, 256, 576), dtype=torch.int16, device=dev)
        out = torch.empty((w.units, 256, 512), dtype=torch.float32, device=dev)
        with pytest.raises(hs.HisparseError) as e:
            hs.hisparse_sparse_decode_noalloc(run.cache.handle, 0, q, run.slots[0], out, big,
                                              run.stream)
        assert e.value.status == hs.HISPARSE_ERR_UNSUPPORTED
        deferred = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, 1, 0, w.scale,
                               hs.HISPARSE_ATTN_DEFER_MERGE)
        with pytest.raises(hs.HisparseError) as e:
            hs.hisparse_sparse_decode_noalloc(run.cache.handle, 0, q, run.slots[0], out,
                                              deferred, run.stream)
        assert e.value.status == hs.HISPARSE_ERR_INVALID_ARG
    finally:
        torch.cuda.synchronize()
        run.close()
