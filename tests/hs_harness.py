"""GPU test harness: drives the HIP library through its C ABI on seeded workloads and checks it
against the CPU oracle. Imported by the GPU tests only."""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle
import workload as W
from paper_2608_07009_amd import HiSparseCache, hisparse as hs


def log(msg: str) -> None:
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def attn_desc(w: W.Workload, num_splits: int = 0, flags: int = 0) -> hs.AttnDesc:
    return hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, num_splits,
                       w.scale, flags)


class Run:
    """One cache for a workload, its host pools filled, selections on the device."""

    def __init__(self, w: W.Workload, steps: int, fill: bool = True,
                 fetch: int = hs.HISPARSE_FETCH_ZERO_COPY, layers_to_fill=None, **kw):
        fitted = W.fit_pinned(w)
        if fitted.num_layers != w.num_layers:
            log(f"{w.name}: host pools of {w.num_layers} layers exceed the pinned budget; "
                f"running {fitted.num_layers} layers")
        w = fitted
        self.w = w
        self.steps = steps
        self.dev = torch.device("cuda:0")
        t0 = time.time()
        self.cache = HiSparseCache.for_workload(w, fetch=fetch, **kw)
        log(f"{w.name}: cache created in {time.time() - t0:.1f}s "
            f"(host {w.host_pool_bytes() / 2**30:.2f} GiB, HBM cache {w.cache_bytes() / 2**20:.0f} MiB)")
        if fill:
            t0 = time.time()
            for l in (range(w.num_layers) if layers_to_fill is None else layers_to_fill):
                ptr, n = self.cache.host_pool(l)
                W.fill_kv(ptr, w, l)
            log(f"{w.name}: host pools filled in {time.time() - t0:.1f}s")
        t0 = time.time()
        self.sel_host = W.selection_streams(w, steps=steps)  # [steps][streams][k]
        self.sel = torch.from_numpy(self.sel_host).to(self.dev)
        log(f"{w.name}: {steps} steps of selections in {time.time() - t0:.1f}s")
        U, k = w.units, w.k
        self.slots = torch.empty((w.num_layers, U, k), dtype=torch.int32, device=self.dev)
        self.counts = torch.empty((w.num_layers, U, 2), dtype=torch.int32, device=self.dev)
        self.stream = torch.cuda.current_stream()

    def sel_ptr(self, step: int, layer: int) -> int:
        a = layer // self.w.share_group
        return self.sel[step, a * self.w.units:(a + 1) * self.w.units].data_ptr()

    def resolve_step(self, step: int, prefetch: bool = False) -> None:
        w = self.w
        for l in w.anchors:
            hs.hisparse_resolve(self.cache.handle, l, self.sel_ptr(step, l), self.slots[l],
                                self.counts[l], self.stream)
            if prefetch:
                for s in range(l + 1, min(l + w.share_group, w.num_layers)):
                    hs.hisparse_prefetch_layer(self.cache.handle, l, s, self.stream)

    def close(self):
        self.cache.close()


_hip = None


def hip():
    """libamdhip64 for raw device copies in the tests."""
    global _hip
    if _hip is None:
        import ctypes
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.restype = ctypes.c_int
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_int]
    return _hip


def d2h(ptr: int, nbytes: int) -> np.ndarray:
    out = np.empty(nbytes, dtype=np.uint8)
    torch.cuda.synchronize()
    rc = hip().hipMemcpy(out.ctypes.data, ptr, nbytes, 2)  # hipMemcpyDeviceToHost
    assert rc == 0, f"hipMemcpy D2H failed ({rc})"
    return out


def layer_cache_host(run: "Run", layer: int) -> np.ndarray:
    """uint8 [units][B][R] copy of a layer's GPU cache."""
    ptr, n = run.cache.layer_cache(layer)
    w = run.w
    return d2h(ptr, n).reshape(w.units, w.B, w.record_bytes)


def expected_order(slot_ts: np.ndarray) -> np.ndarray:
    """Slots of each unit by ascending (timestamp, slot)."""
    B = slot_ts.shape[-1]
    return np.stack([np.lexsort((np.arange(B), ts)) for ts in slot_ts]).astype(np.int32)


def turn_step(runs, streams, turns, t, n_layers):
    """One step of two or more micro-batches taking device link turns: the turns reset on the
    first stream, the others forked from it, then per layer each micro-batch's resolve and its
    fetch waiting for the previous micro-batch's turn; joined back into the first stream."""
    n_mb = len(runs)
    hs.hisparse_link_turns_reset(turns, n_layers * n_mb, streams[0])
    fork = torch.cuda.Event()
    fork.record(streams[0])
    for s in streams[1:]:
        s.wait_event(fork)
    for l in range(n_layers):
        for i, (r, s) in enumerate(zip(runs, streams)):
            hs.hisparse_resolve_tables(r.cache.handle, l, r.sel_ptr(t, l), r.slots[l],
                                       r.counts[l], s)
            ti = l * n_mb + i
            hs.hisparse_fetch_turn(r.cache.handle, l, turns, n_layers * n_mb, ti - 1, ti, 192,
                                   s)
    for s in streams[1:]:
        j = torch.cuda.Event()
        j.record(s)
        streams[0].wait_event(j)
