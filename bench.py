#!/usr/bin/env python3
"""Benchmark of the HiSparse decode hot path on one MI355X.

One step = one decode step of every layer: resolve (phases 1-3, 5) + miss fetch (phase 4) for
each anchor layer, exact-prefetch replays for shared layers (side stream), and sparse decode
attention for every layer, over seeded synthetic inputs already resident in HBM / pinned host
memory. Default workload: 32 requests x 8 layers, 32K-token context, k=2048, B=4096 slots,
128 latent-attention heads.

Prints one JSON line: value = selections served per second (layers x units x k per step over
wall time), with the miss-fetch GB/s against the in-process pinned hipMemcpy H2D peak, decode
tokens/s, per-kernel event timings, the roofline of the dominant kernel and the CPU oracle
baseline.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, published
PCIE_PEAK_GBPS = 64.0           # PCIe Gen5 x16, one direction, published host interface


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--fetch", choices=["zero_copy", "none"], default="zero_copy")
    ap.add_argument("--host-memory", choices=["coherent", "noncoherent", "uncached"],
                    default="coherent")
    ap.add_argument("--transfer-block", type=int, default=0)
    ap.add_argument("--splits", type=int, default=0, help="attention splits (0 = auto)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work")
    ap.add_argument("--no-sweep", action="store_true")
    return ap.parse_args()


class Hip:
    """Raw hipMemcpyAsync for the pinned H2D sweep."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipMemcpyAsync.restype = ctypes.c_int
        self.lib.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                            ctypes.c_int, ctypes.c_void_p]

    def h2d_async(self, dst: int, src: int, n: int, stream: int) -> None:
        rc = self.lib.hipMemcpyAsync(dst, src, n, 1, stream)  # hipMemcpyHostToDevice
        if rc != 0:
            raise RuntimeError(f"hipMemcpyAsync failed ({rc})")


def pinned_sweep(torch, host_ptr: int, host_bytes: int, dev, stream) -> dict:
    """H2D bandwidth of hipMemcpyAsync from the library's pinned pool, 4 KiB .. 1 GiB."""
    hip = Hip()
    top = min(1 << 30, host_bytes)
    dst = torch.empty(top, dtype=torch.uint8, device=dev)
    res = {}
    size = 4096
    while size <= top:
        reps = max(3, min(2000, (256 << 20) // size))
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        hip.h2d_async(dst.data_ptr(), host_ptr, size, stream.cuda_stream)  # warm
        s.record(stream)
        for _ in range(reps):
            hip.h2d_async(dst.data_ptr(), host_ptr, size, stream.cuda_stream)
        e.record(stream)
        e.synchronize()
        res[size] = size * reps / (s.elapsed_time(e) * 1e-3) / 1e9
        size *= 4
    del dst
    return res


class Events:
    """Per-kernel HIP event pairs recorded on the kernel's own stream."""

    def __init__(self, torch):
        self.torch = torch
        self.spans = []  # (name, start, end)

    def span(self, name, stream, fn):
        s = self.torch.cuda.Event(enable_timing=True)
        e = self.torch.cuda.Event(enable_timing=True)
        s.record(stream)
        fn()
        e.record(stream)
        self.spans.append((name, s, e))

    def totals(self) -> dict:
        out = {}
        for name, s, e in self.spans:
            t, n = out.get(name, (0.0, 0))
            out[name] = (t + s.elapsed_time(e) * 1e-3, n + 1)
        return out


def cpu_baseline(w, cache, sel_host, budget_s: float) -> dict:
    """The oracle, as it stands, on a bounded sample: resolve + gather + float64 attention of
    units of layer 0, steps from cold, until the time budget is used."""
    import numpy as np

    import oracle
    import workload as W

    n_units = min(4, w.units)
    orcs = [oracle.OracleCache(1, w.L, w.B, w.k) for _ in range(n_units)]
    imgs = [np.zeros((w.B, w.record_bytes), dtype=np.uint8) for _ in range(n_units)]
    host = cache.host_view(0)
    done = 0
    t0 = time.perf_counter()
    t = 0
    while time.perf_counter() - t0 < budget_s and t < sel_host.shape[0]:
        q = W.queries(w, t, 0, 0, n_units)
        for u in range(n_units):
            rc, slots, counts, pp, ps = orcs[u].resolve_unit(0, sel_host[t, u])
            oracle.apply_plan(host[u], imgs[u], pp, ps)
            oracle.sparse_decode(q[u], imgs[u].view(np.uint16).reshape(w.B, -1), slots,
                                 d_qk=w.d_qk, d_v=w.d_v, v_off=w.v_offset,
                                 token_elems=w.token_elems,
                                 tokens_per_record=w.tokens_per_record, scale=w.scale)
            done += 1
        t += 1
    dt = time.perf_counter() - t0
    return {"value": done * w.k / dt, "unit": "selections/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} unit-steps (units 0..{n_units - 1} of layer 0, steps 0..{t - 1} "
                      f"from cold): canonical-LRU resolve + record gather + float64 attention "
                      f"over {w.q_heads} heads, single thread, {dt:.1f} s"}


def main() -> int:
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: HiSparse's units "
                          "are independent caches, so more GPUs shard requests without any "
                          "exchange; run one process per GPU", "n_gpus": args.gpus}))
        return 2

    import numpy as np
    import torch

    import workload as W
    from paper_2608_07009_amd import HiSparseCache, hisparse as hs

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        return 1
    hs.lib()  # fails loudly if the HIP library is missing
    w0 = W.workload(args.config)
    w = W.fit_pinned(w0)
    steps_needed = args.warmup + args.steps
    if steps_needed > w.steps:
        print(json.dumps({"error": f"warmup + steps = {steps_needed} exceeds the workload's "
                          f"{w.steps} steps"}))
        return 2
    dev = torch.device("cuda:0")
    main_s = torch.cuda.current_stream()
    side_s = torch.cuda.Stream()
    fetch = hs.HISPARSE_FETCH_NONE if args.fetch == "none" else hs.HISPARSE_FETCH_ZERO_COPY
    hmem = {"coherent": hs.HISPARSE_HOST_COHERENT, "noncoherent": hs.HISPARSE_HOST_NONCOHERENT,
            "uncached": hs.HISPARSE_HOST_UNCACHED}[args.host_memory]

    t0 = time.time()
    cache = HiSparseCache.for_workload(w, fetch=fetch, host_memory=hmem,
                                       transfer_block_bytes=args.transfer_block)
    for l in range(w.num_layers):
        W.fill_kv(cache.host_pool(l)[0], w, l)
    sel_host = W.selection_streams(w, steps=steps_needed)
    sel = torch.from_numpy(sel_host).to(dev)
    n_qv = 2  # queries vary by (layer, step parity)
    q_all = torch.stack([torch.stack([torch.from_numpy(W.queries(w, v, l).view(np.int16))
                                      for l in range(w.num_layers)]) for v in range(n_qv)]).to(dev)
    log(f"{w.name}: layers {w.num_layers} (of {w0.num_layers}), host pool "
        f"{w.host_pool_bytes() / 2**30:.1f} GiB, set up in {time.time() - t0:.1f}s")

    U, k = w.units, w.k
    slots = torch.empty((w.num_layers, U, k), dtype=torch.int32, device=dev)
    counts = torch.zeros((steps_needed, w.num_layers, U, 2), dtype=torch.int32, device=dev)
    ad = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, args.splits,
                     w.scale, 0)
    ws_bytes = hs.hisparse_decode_workspace_bytes(U, k, w.record_bytes, ad)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((w.num_layers, U, w.q_heads, w.d_v), dtype=torch.float32, device=dev)
    h = cache.handle
    G = w.share_group

    def step(t: int, ev: Events | None):
        def span(name, stream, fn):
            if ev is None:
                fn()
            else:
                ev.span(name, stream, fn)

        qv = q_all[t % n_qv]
        for a in w.anchors:
            ai = a // G
            sel_a = sel[t, ai * U:(ai + 1) * U]
            span("resolve_tables", main_s,
                 lambda: hs.hisparse_resolve_tables(h, a, sel_a, slots[a], counts[t, a], main_s))
            shared = list(range(a + 1, min(a + G, w.num_layers)))
            done = {}
            if shared:
                fork = torch.cuda.Event()
                fork.record(main_s)
                side_s.wait_event(fork)
                for s in shared:
                    span("prefetch_replay", side_s,
                         lambda s=s: hs.hisparse_prefetch_layer(h, a, s, side_s))
                    done[s] = torch.cuda.Event()
                    done[s].record(side_s)
            span("fetch", main_s, lambda: hs.hisparse_fetch(h, a, main_s))
            span("sparse_decode", main_s,
                 lambda: hs.hisparse_sparse_decode(h, a, qv[a], slots[a], out[a], ad, ws,
                                                   ws_bytes, main_s))
            for s in shared:
                main_s.wait_event(done[s])
                span("sparse_decode", main_s,
                     lambda s=s: hs.hisparse_sparse_decode(h, s, qv[s], slots[a], out[s], ad, ws,
                                                           ws_bytes, main_s))

    # pinned H2D sweep over the same pool (hipMemcpyAsync), before the timed region
    sweep = {}
    if not args.no_sweep:
        sweep = pinned_sweep(torch, *cache.host_pool(0), dev, main_s)
        log("pinned H2D sweep GB/s: " + ", ".join(f"{s >> 10}K:{v:.1f}" for s, v in sweep.items()))
    pinned_peak = max(sweep.values()) if sweep else None

    # warmup (step 0 is the cold step)
    torch.cuda.synchronize()
    tc = time.perf_counter()
    step(0, None)
    torch.cuda.synchronize()
    cold_ms = (time.perf_counter() - tc) * 1e3
    for t in range(1, args.warmup):
        step(t, None)
    torch.cuda.synchronize()

    # timed region
    ev = Events(torch)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.warmup, steps_needed):
        step(t, ev)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st, info = cache.check_errors()
    if st != hs.HISPARSE_OK:
        print(json.dumps({"error": f"device-side selection error {info}"}))
        return 1

    tot = ev.totals()
    c = counts[args.warmup:steps_needed].cpu().numpy().astype(np.int64)  # [K][layers][U][2]
    K = args.steps
    anchor_calls = K * len(w.anchors)
    misses_anchor = int(c[:, w.anchors, :, 1].sum())
    hits_anchor = int(c[:, w.anchors, :, 0].sum())
    shared_per_anchor = {a: len(range(a + 1, min(a + G, w.num_layers))) for a in w.anchors}
    misses_replay = int(sum(c[:, a, :, 1].sum() * n for a, n in shared_per_anchor.items()))
    R = w.record_bytes
    served = K * w.num_layers * U * k
    value = served / wall

    def kernel(name):
        t, n = tot.get(name, (0.0, 0))
        return t, n

    t_tab, n_tab = kernel("resolve_tables")
    t_fet, n_fet = kernel("fetch")
    t_rep, n_rep = kernel("prefetch_replay")
    t_att, n_att = kernel("sparse_decode")
    fetch_bytes = misses_anchor * R
    replay_bytes = misses_replay * R
    kernels = {}
    # resolve tables: integer metadata work per unit (algorithmic bytes):
    # sel 4k + page-table probes 4k + slot outputs 4k + recency index read+write 8B
    # + hit stamps 4h + per miss (slot map r/w 8, page table 8, stamp 4, plan 8) = 28m
    tab_bytes = anchor_calls * U * (12 * k + 8 * w.B) + 4 * hits_anchor + 28 * misses_anchor
    if n_tab:
        kernels["resolve_tables"] = {
            "launches": n_tab, "avg_us": t_tab / n_tab * 1e6, "bound": "latency",
            "hbm_GBps": tab_bytes / t_tab / 1e9,
            "selections_per_s_no_io": anchor_calls * U * k / t_tab}
    if n_fet and fetch != hs.HISPARSE_FETCH_NONE:
        kernels["fetch"] = {"launches": n_fet, "avg_us": t_fet / n_fet * 1e6,
                            "bytes_per_launch": fetch_bytes / n_fet,
                            "GBps": fetch_bytes / t_fet / 1e9}
    if n_rep and fetch != hs.HISPARSE_FETCH_NONE:
        kernels["prefetch_replay"] = {"launches": n_rep, "avg_us": t_rep / n_rep * 1e6,
                                      "bytes_per_launch": replay_bytes / n_rep,
                                      "GBps": replay_bytes / t_rep / 1e9}
    n_tok = k * w.tokens_per_record
    att_flops_call = 2.0 * U * w.q_heads * n_tok * (w.d_qk + w.d_v)
    att_bytes_call = (U * n_tok * (R // w.tokens_per_record) + U * w.q_heads * w.d_qk * 2
                      + U * w.q_heads * w.d_v * 4 + U * k * 4)
    if n_att:
        a_time = t_att / n_att
        kernels["sparse_decode"] = {
            "launches": n_att, "avg_us": a_time * 1e6,
            "bytes_per_launch": att_bytes_call, "flops_per_launch": att_flops_call,
            "hbm_GBps": att_bytes_call / a_time / 1e9,
            "mfma_TFLOPs": att_flops_call / a_time / 1e12,
            "hbm_frac": att_bytes_call / a_time / 1e9 / HBM_PEAK_GBPS,
            "mfma_frac": att_flops_call / a_time / 1e12 / MFMA_BF16_PEAK_TFLOPS}

    # dominant kernel by total event time
    totals = {"resolve_tables": t_tab, "fetch": t_fet, "prefetch_replay": t_rep,
              "sparse_decode": t_att}
    dom = max(totals, key=totals.get)
    if dom in ("fetch", "prefetch_replay"):
        kd = kernels[dom]
        roof = {"kernel": dom, "bound": "host_link", "achieved": kd["GBps"],
                "peak": PCIE_PEAK_GBPS, "unit": "GB/s", "frac": kd["GBps"] / PCIE_PEAK_GBPS,
                "traffic": None, "measured_pinned_h2d_peak": pinned_peak,
                "frac_of_measured_peak": (kd["GBps"] / pinned_peak) if pinned_peak else None,
                "algorithmic_bytes_per_launch": kd["bytes_per_launch"]}
    elif dom == "sparse_decode":
        kd = kernels[dom]
        t_hbm = att_bytes_call / (HBM_PEAK_GBPS * 1e9)
        t_mfma = att_flops_call / (MFMA_BF16_PEAK_TFLOPS * 1e12)
        if t_hbm >= t_mfma:
            roof = {"kernel": dom, "bound": "hbm", "achieved": kd["hbm_GBps"],
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": kd["hbm_frac"]}
        else:
            roof = {"kernel": dom, "bound": "mfma", "achieved": kd["mfma_TFLOPs"],
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": kd["mfma_frac"]}
        roof.update({"traffic": None, "algorithmic_bytes_per_launch": att_bytes_call,
                     "flops_per_launch": att_flops_call})
    else:
        kd = kernels["resolve_tables"]
        roof = {"kernel": dom, "bound": "hbm", "achieved": kd["hbm_GBps"], "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": kd["hbm_GBps"] / HBM_PEAK_GBPS, "traffic": None}

    miss_gbps = (fetch_bytes + replay_bytes) / (t_fet + t_rep) / 1e9 if (t_fet + t_rep) else None
    result = {
        "metric": "resolved selections/s + miss-fetch GB/s (% host-link peak), decode tokens/s",
        "value": value,
        "unit": "selections/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": wall / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32+bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "requests": w.num_requests, "layers": w.num_layers,
                   "layers_in_workload": w0.num_layers, "units_per_layer": U,
                   "records_per_unit": w.L, "record_bytes": R, "top_k": k, "capacity": w.B,
                   "share_group": G, "q_heads": w.q_heads, "fetch": args.fetch,
                   "host_memory": args.host_memory, "mode": "eager"},
        "decode_tokens_per_s": w.num_requests * K / wall,
        "miss_fetch_GBps": miss_gbps,
        "miss_fetch_pct_of_pinned_h2d_peak": (100 * miss_gbps / pinned_peak)
        if (miss_gbps and pinned_peak) else None,
        "pinned_h2d_peak_GBps": pinned_peak,
        "pinned_h2d_sweep_GBps": {str(s): v for s, v in sweep.items()},
        "hit_rate": hits_anchor / max(1, hits_anchor + misses_anchor),
        "misses_per_unit_step": misses_anchor / max(1, anchor_calls * U),
        "cold_step_ms": cold_ms,
        "kernels": kernels,
        "roofline": roof,
        "hbm_footprint_GiB": (w0.num_layers * U * w.B * R) / 2**30,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(w, cache, sel_host[:, :U], args.cpu_budget)
    cache.close()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
