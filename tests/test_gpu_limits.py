"""GPU parity at the limits a cache descriptor accepts.

  * the largest slot count and top-k (B = 16384, k = 4096) over enough steps that the cache
    fills and evicts, with padding in one step: slots, counts and every table against the
    oracle, bit-exact, and every resident slot holding its record;
  * the smallest record (16 B, one transfer block) and a large one (64 KiB): resident bytes;
  * the widest latent attention (256 heads) over the largest top-k: the cache path equals the
    fully resident path bit for bit and the oracle within tolerance on sampled heads;
  * the degenerate cache sizes B = k and B = L, with their closed forms.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workload as W
from hs_harness import attn_desc, d2h, expected_order, log
from paper_2608_07009_amd import HiSparseCache, hisparse as hs

pytestmark = pytest.mark.gpu

MAX_ABS, REL_L2 = 1e-2, 5e-3


def carried_stream(rng, steps, U, L, k, keep):
    """int32 [steps][U][k]: distinct positions; a fraction `keep` of each step's set carried
    from the previous step, the rest fresh; shuffled."""
    out = np.empty((steps, U, k), dtype=np.int32)
    for u in range(U):
        prev = rng.choice(L, size=k, replace=False)
        out[0, u] = prev
        for t in range(1, steps):
            kept = rng.choice(prev, size=int(keep * k), replace=False)
            pool = np.setdiff1d(np.arange(L), prev)
            fresh = rng.choice(pool, size=k - len(kept), replace=False)
            prev = rng.permutation(np.concatenate([kept, fresh]))
            out[t, u] = prev
    return out


def check_resident(cache, layer, orc, U, B, R, host):
    ptr, n = cache.layer_cache(layer)
    dev = d2h(ptr, n).reshape(U, B, R)
    for u in range(U):
        res = np.nonzero(orc.slot_pos[u] >= 0)[0]
        assert (dev[u][res] == host[u][orc.slot_pos[u][res]]).all(), f"unit {u}"


def test_resolve_at_maximum_capacity_and_topk():
    U, L, B, k, R, steps = 2, 65536, 16384, 4096, 64, 16
    log(f"test_resolve_at_maximum_capacity_and_topk U={U} L={L} B={B} k={k} steps={steps}")
    rng = np.random.default_rng(91)
    sel = carried_stream(rng, steps, U, L, k, keep=0.7)
    sel[5, 1, ::7] = -1  # padding entries in one step of one unit
    cache = HiSparseCache(num_requests=U, num_layers=1, units_per_request=1, capacity=B,
                          num_records=L, top_k=k, record_bytes=R)
    try:
        host = cache.host_view(0)
        host[:] = rng.integers(0, 256, size=host.shape, dtype=np.uint8)
        dev = torch.device("cuda:0")
        stream = torch.cuda.current_stream()
        sel_d = torch.from_numpy(sel).to(dev)
        slots = torch.empty((U, k), dtype=torch.int32, device=dev)
        counts = torch.empty((U, 2), dtype=torch.int32, device=dev)
        orc = oracle.OracleCache(U, L, B, k)
        evicted = False
        for t in range(steps):
            hs.hisparse_resolve(cache.handle, 0, sel_d[t], slots, counts, stream)
            torch.cuda.synchronize()
            e_slots, e_counts, _, _, bad = orc.resolve(sel[t])
            assert bad == 0
            assert (slots.cpu().numpy() == e_slots).all(), f"slots step {t}"
            assert (counts.cpu().numpy() == e_counts).all(), f"counts step {t}"
            evicted = evicted or bool((orc.slot_pos >= 0).sum() == U * B)
        assert evicted, "the cache never filled: no eviction was exercised"
        assert cache.check_errors()[0] == hs.HISPARSE_OK
        st = cache.read_state(0)
        assert (st["slot_pos"] == orc.slot_pos).all()
        assert (st["slot_ts"] == orc.slot_ts).all()
        assert (st["clock"] == orc.clock).all()
        assert (st["page_table"] == orc.pt).all()
        assert (st["order"] == expected_order(orc.slot_ts)).all()
        check_resident(cache, 0, orc, U, B, R, host)
    finally:
        torch.cuda.synchronize()
        cache.close()


@pytest.mark.parametrize("R", [16, 65536])
def test_fetch_smallest_and_large_records(R):
    U, L, B, k, steps = 3, 512, 256, 128, 5
    log(f"test_fetch_smallest_and_large_records R={R}")
    rng = np.random.default_rng(92 + R)
    sel = carried_stream(rng, steps, U, L, k, keep=0.5)
    cache = HiSparseCache(num_requests=U, num_layers=1, units_per_request=1, capacity=B,
                          num_records=L, top_k=k, record_bytes=R)
    try:
        host = cache.host_view(0)
        host[:] = rng.integers(0, 256, size=host.shape, dtype=np.uint8)
        dev = torch.device("cuda:0")
        sel_d = torch.from_numpy(sel).to(dev)
        slots = torch.empty((U, k), dtype=torch.int32, device=dev)
        orc = oracle.OracleCache(U, L, B, k)
        for t in range(steps):
            hs.hisparse_resolve(cache.handle, 0, sel_d[t], slots, None,
                                torch.cuda.current_stream())
            torch.cuda.synchronize()
            e_slots, _, _, _, _ = orc.resolve(sel[t])
            assert (slots.cpu().numpy() == e_slots).all(), f"slots step {t}"
            check_resident(cache, 0, orc, U, B, R, host)
    finally:
        torch.cuda.synchronize()
        cache.close()


def test_attention_widest_mla_at_maximum_topk():
    w = dataclasses.replace(W.workload(2), num_requests=1, num_layers=1, q_heads=256, k=4096,
                            B=4096, L=8192, window=64, carry=0)
    log(f"test_attention_widest_mla_at_maximum_topk H={w.q_heads} k={w.k}")
    rng = np.random.default_rng(93)
    cache = HiSparseCache.for_workload(w)
    try:
        dev = torch.device("cuda:0")
        host = cache.host_view(0)
        W.fill_kv(cache.host_pool(0)[0], w, 0)
        sel = rng.choice(w.L, size=(1, w.k), replace=False).astype(np.int32)
        sel_d = torch.from_numpy(sel).to(dev)
        slots = torch.empty((1, w.k), dtype=torch.int32, device=dev)
        hs.hisparse_resolve(cache.handle, 0, sel_d, slots, None, torch.cuda.current_stream())
        q_host = W.queries(w, 0, 0)
        q = torch.from_numpy(q_host.view(np.int16)).to(dev)
        ad = attn_desc(w)
        nb = hs.hisparse_decode_workspace_bytes(1, w.k, w.record_bytes, ad)
        ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        out_c = torch.empty((1, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
        out_r = torch.empty_like(out_c)
        hs.hisparse_sparse_decode(cache.handle, 0, q, slots, out_c, ad, ws, nb,
                                  torch.cuda.current_stream())
        resident = torch.from_numpy(host.reshape(-1)).to(dev)
        hs.hisparse_sparse_decode_pool(resident, w.L, w.record_bytes, 1, w.k, q, sel_d, out_r,
                                       ad, ws, nb, torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(out_c, out_r)
        heads = [0, 31, 32, 127, 128, 255]
        pool_u = host[0].view(np.uint16).reshape(w.L, -1)
        ref = oracle.sparse_decode(q_host[0][heads], pool_u, sel[0], d_qk=w.d_qk, d_v=w.d_v,
                                   v_off=w.v_offset, token_elems=w.token_elems,
                                   tokens_per_record=w.tokens_per_record, scale=w.scale)
        o = out_c.cpu().numpy()[0][heads]
        err, rl2 = np.abs(o - ref).max(), float(np.linalg.norm(o - ref) / np.linalg.norm(ref))
        log(f"  max-abs {err:.2e} rel-L2 {rl2:.2e}")
        assert err <= MAX_ABS and rl2 <= REL_L2
    finally:
        torch.cuda.synchronize()
        cache.close()


@pytest.mark.parametrize("B,L", [(128, 4096), (512, 512)])
def test_resolve_degenerate_cache_sizes(B, L):
    """B = k: the cache holds exactly the step's selection (every non-selected record is
    evicted at once); B = L: nothing is ever evicted. Bit-exact against the oracle, with the
    closed forms of both cases checked on the GPU's own counts."""
    U, k, R, steps = 3, 128, 32, 12
    log(f"test_resolve_degenerate_cache_sizes B={B} L={L} k={k}")
    rng = np.random.default_rng(94 + B)
    sel = carried_stream(rng, steps, U, L, k, keep=0.6)
    cache = HiSparseCache(num_requests=U, num_layers=1, units_per_request=1, capacity=B,
                          num_records=L, top_k=k, record_bytes=R)
    try:
        host = cache.host_view(0)
        host[:] = rng.integers(0, 256, size=host.shape, dtype=np.uint8)
        dev = torch.device("cuda:0")
        sel_d = torch.from_numpy(sel).to(dev)
        slots = torch.empty((U, k), dtype=torch.int32, device=dev)
        counts = torch.empty((U, 2), dtype=torch.int32, device=dev)
        orc = oracle.OracleCache(U, L, B, k)
        seen = [set() for _ in range(U)]
        for t in range(steps):
            hs.hisparse_resolve(cache.handle, 0, sel_d[t], slots, counts,
                                torch.cuda.current_stream())
            torch.cuda.synchronize()
            e_slots, e_counts, _, _, _ = orc.resolve(sel[t])
            got = counts.cpu().numpy()
            assert (slots.cpu().numpy() == e_slots).all(), f"slots step {t}"
            assert (got == e_counts).all(), f"counts step {t}"
            for u in range(U):
                cur = set(sel[t, u].tolist())
                if B == k:  # top-k staging: misses = |S_t minus S_(t-1)|
                    prev = set(sel[t - 1, u].tolist()) if t else set()
                    assert got[u, 1] == len(cur - prev)
                else:  # no eviction: misses = first touches only
                    assert got[u, 1] == len(cur - seen[u])
                seen[u] |= cur
            check_resident(cache, 0, orc, U, B, R, host)
        st = cache.read_state(0)
        assert (st["page_table"] == orc.pt).all() and (st["slot_ts"] == orc.slot_ts).all()
    finally:
        torch.cuda.synchronize()
        cache.close()
