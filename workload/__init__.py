"""Seeded synthetic workloads for the HiSparse decode hot path.

Shared input infrastructure: the five workload shapes, and ctypes access to the C generator
(`hs_workload.c`) that draws KV records, decode queries and top-k selection streams. Nothing
here implements residency, replacement or attention; the GPU library and the CPU oracle both
consume these inputs.

Shapes follow the paper's evaluated families (Section 4.1 "Setup": DSA token-level top-2048,
NSA-style block selection, Quest page selection; BF16 KV) and its design sizes (Section 3.2:
B slots per request and layer, B >= k; Section 3.5: shared selections across groups of four
layers). The selection law (window + carried subset + Zipf/Gumbel fresh draws) is a synthetic
stand-in for the paper's LongBenchV2 selection trace, which is not available.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_DIR = os.path.join(_HERE, "lib")
_LIB_PATH = os.path.join(_LIB_DIR, "libhs_workload.so")
_SRC = os.path.join(_HERE, "hs_workload.c")


def build(force: bool = True, path: str | None = None, extra_flags=()) -> str:
    """Compile the generator with gcc into workload/lib/libhs_workload.so, or into `path` with
    extra compiler flags (e.g. a sanitizer build)."""
    out = path or _LIB_PATH
    os.makedirs(os.path.dirname(out), exist_ok=True)
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-Wall", "-Wextra", "-Wno-unused-parameter", *extra_flags,
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, out)
    return out


class _StreamParams(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int64), ("k", ctypes.c_int32), ("window", ctypes.c_int32),
                ("carry", ctypes.c_int32), ("steps", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("zipf_s", ctypes.c_double), ("drift", ctypes.c_double),
                ("seed", ctypes.c_uint64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("HS_WORKLOAD_LIB") or _LIB_PATH  # another build, e.g. sanitized
        if not os.path.exists(path):
            raise RuntimeError("workload generator not built: run __graft_entry__.build()")
        L = ctypes.CDLL(path)
        L.hs_key.restype = ctypes.c_uint64
        L.hs_key.argtypes = [ctypes.c_uint64] * 5
        L.hs_splitmix64.restype = ctypes.c_uint64
        L.hs_splitmix64.argtypes = [ctypes.c_uint64]
        L.hs_normal_table.restype = ctypes.POINTER(ctypes.c_uint16)
        L.hs_fill_kv.restype = ctypes.c_int
        L.hs_fill_kv.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64,
                                 ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                 ctypes.c_int32]
        L.hs_fill_q.restype = ctypes.c_int
        L.hs_fill_q.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32]
        L.hs_gen_streams.restype = ctypes.c_int
        L.hs_gen_streams.argtypes = [ctypes.POINTER(_StreamParams), ctypes.c_int64,
                                     ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32]
        _lib = L
    return _lib


def default_threads() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return max(1, min(16, n or 1))


@dataclass(frozen=True)
class Workload:
    """One synthetic decode workload. A *unit* is one independent cache: a (request, layer)
    for token-level DSA/MLA, a (request, layer, kv head) for NSA/Quest."""
    name: str
    num_requests: int
    num_layers: int
    units_per_request: int
    L: int                 # records per unit (tokens, 64-token blocks, 16-token pages)
    record_bytes: int      # R
    k: int                 # selected records per unit per step
    B: int                 # cache slots per unit
    share_group: int       # 1: every layer selects; 4: anchors at layer % 4 == 0
    steps: int
    window: int            # last `window` records always selected
    carry: int             # records carried from the previous step's non-window part
    kind: int              # 0 Zipf over a drifting permutation, 1 Gumbel top-n
    zipf_s: float
    drift: float
    attn: str              # "mla" or "gqa"
    q_heads: int           # query heads per unit
    d_qk: int
    d_v: int
    v_offset: int          # element offset of V inside a token
    tokens_per_record: int
    scale: float
    seed: int

    @property
    def units(self) -> int:
        return self.num_requests * self.units_per_request

    @property
    def token_elems(self) -> int:
        return self.record_bytes // 2 // self.tokens_per_record

    @property
    def record_elems(self) -> int:
        return self.record_bytes // 2

    @property
    def anchors(self) -> list[int]:
        return list(range(0, self.num_layers, self.share_group))

    @property
    def n_streams(self) -> int:
        return len(self.anchors) * self.units

    def stream_params(self) -> _StreamParams:
        return _StreamParams(self.L, self.k, self.window, self.carry, self.steps, self.kind,
                             self.zipf_s, self.drift, self.seed)

    def host_pool_bytes(self) -> int:
        return self.num_layers * self.units * self.L * self.record_bytes

    def cache_bytes(self) -> int:
        return self.num_layers * self.units * self.B * self.record_bytes


MLA_SCALE = 1.0 / math.sqrt(192.0)
GQA_SCALE = 1.0 / math.sqrt(128.0)

WORKLOADS = {
    # 1 request, 1 layer, 4096 tokens, 576-elem records, B=512, k=128, 64 steps
    1: Workload("tiny_dsa_L4096_k128_B512", 1, 1, 1, 4096, 1152, 128, 512, 1, 64,
                32, 0, 0, 1.1, 1.0, "mla", 16, 576, 512, 0, 1, MLA_SCALE, 20261201),
    # 32 requests x 8 layers, 32K tokens, k=2048, B=4096, 128 heads, 256 steps, ~80% overlap
    2: Workload("dsa_mla_32req_8L_ctx32K_k2048_B4096", 32, 8, 1, 32768, 1152, 2048, 4096, 1,
                256, 64, 1587, 0, 1.0, 0.0, "mla", 128, 576, 512, 0, 1, MLA_SCALE, 20261202),
    # 16 requests x 4 kv heads x 8 layers, 128K tokens as 2048 64-token blocks, k=16+8 blocks
    3: Workload("nsa_blocks_16req_4kvh_8L_ctx128K", 16, 8, 4, 2048, 32768, 24, 48, 1, 128,
                8, 11, 1, 0.0, 0.0, "gqa", 16, 128, 128, 128, 64, GQA_SCALE, 20261203),
    # 8 requests x 8 kv heads x 8 layers, 128K tokens as 8192 16-token pages, k=256 pages
    4: Workload("quest_pages_8req_8kvh_8L_ctx128K", 8, 8, 8, 8192, 8192, 256, 384, 1, 128,
                0, 154, 0, 1.2, 0.0, "gqa", 4, 128, 128, 128, 16, GQA_SCALE, 20261204),
    # one 1M-token request, 61 layers sharing selections in groups of 4, k=2048, B=4096
    5: Workload("stress_1M_61L_share4_k2048_B4096", 1, 61, 1, 1048576, 1152, 2048, 4096, 4, 64,
                0, 1024, 0, 0.0, 0.0, "mla", 128, 576, 512, 0, 1, MLA_SCALE, 20261205),
}


def workload(n: int, **overrides) -> Workload:
    w = WORKLOADS[n]
    return replace(w, **overrides) if overrides else w


def selection_streams(w: Workload, steps: int | None = None, nthreads: int | None = None,
                      stream0: int = 0, n_streams: int | None = None) -> np.ndarray:
    """int32 [steps][n_streams][k]; stream id = anchor_index * units + unit."""
    p = w.stream_params()
    if steps is not None:
        p.steps = steps
    ns = w.n_streams - stream0 if n_streams is None else n_streams
    out = np.empty((p.steps, ns, w.k), dtype=np.int32)
    rc = lib().hs_gen_streams(ctypes.byref(p), stream0, ns, out.ctypes.data,
                              nthreads or default_threads())
    if rc != 0:
        raise RuntimeError(f"hs_gen_streams failed ({rc})")
    return out


def grow_streams(w: Workload, sel: np.ndarray) -> np.ndarray:
    """Selections of a context that grows by one record per step (the write-through decode
    loop): positions [0, L) are the prefill, and the record generated at step t sits at L + t.
    The window [L - W, L) of step t becomes [L - W + t, L + t), so every step selects the
    records appended in the previous W steps; drawn entries (all below L - W) are unchanged.
    sel: int32 [steps][streams][k] from selection_streams."""
    out = np.array(sel, dtype=np.int32, copy=True)
    if w.window > 0:
        t = np.arange(out.shape[0], dtype=np.int32).reshape(-1, 1, 1)
        out = np.where(out >= w.L - w.window, out + t, out).astype(np.int32)
    return out


def correlate_layers(w: Workload, sel: np.ndarray, rho: float, seed: int = 0) -> np.ndarray:
    """Selections of adjacent layers that overlap within a step (the cross-layer locality that
    a speculative hint from layer l to layer l+1 relies on), keeping each layer's overlap
    across steps. For anchor i >= 1 a seeded mask marks a fraction rho of the positions below
    the window [L - W, L) as taken from anchor i-1: at every step anchor i selects its own
    window, anchor i-1's (already correlated) drawn entries at marked positions, and its own
    drawn entries at unmarked positions; the count is brought back to k by dropping random
    own entries or adding its own entries at marked positions (then random unselected
    positions). The mask is fixed per layer, so entries that persist across steps in either
    layer keep persisting. The set is emitted in shuffled order. sel: int32
    [steps][anchors * units][k] without padding."""
    out = np.array(sel, dtype=np.int32, copy=True)
    if rho <= 0:
        return out
    rng = np.random.default_rng(seed)
    U, lo, k = w.units, w.L - w.window, w.k
    for i in range(1, out.shape[1] // U):
        marked = rng.random(w.L) < rho
        marked[lo:] = False
        for t in range(out.shape[0]):
            for u in range(U):
                prev, own = out[t, (i - 1) * U + u], sel[t, i * U + u]
                if (own < 0).any():
                    raise ValueError("correlate_layers expects selections without padding")
                win = own[own >= lo]
                a = prev[(prev >= 0) & (prev < lo)]
                a = a[marked[a]]
                b = own[(own < lo) & ~marked[np.minimum(own, w.L - 1)]]
                need = k - len(win)
                if len(a) + len(b) > need:
                    drop = len(a) + len(b) - need
                    if drop <= len(b):
                        b = np.delete(b, rng.choice(len(b), drop, replace=False))
                    else:
                        a = np.delete(a, rng.choice(len(a), drop - len(b), replace=False))
                        b = b[:0]
                fill = need - len(a) - len(b)
                c = own[(own < lo) & marked[np.minimum(own, w.L - 1)]]
                c = c[~np.isin(c, a)][:fill]
                parts = [win, a, b, c]
                short = fill - len(c)
                if short > 0:
                    used = np.concatenate(parts)
                    pool = np.setdiff1d(np.arange(lo, dtype=np.int32), used)
                    parts.append(rng.choice(pool, short, replace=False).astype(np.int32))
                out[t, i * U + u] = rng.permutation(np.concatenate(parts))
    return out


def fill_kv(ptr: int, w: Workload, layer: int, unit0: int = 0, n_units: int | None = None,
            rec0: int = 0, n_rec: int | None = None, nthreads: int | None = None) -> None:
    """Write records [unit0, unit0+n_units) x [rec0, rec0+n_rec) of `layer` to raw memory `ptr`
    laid out [unit][record][record_elems] bf16."""
    nu = w.units - unit0 if n_units is None else n_units
    nr = w.L - rec0 if n_rec is None else n_rec
    rc = lib().hs_fill_kv(ctypes.c_void_p(ptr), w.seed, layer, unit0, nu, rec0, nr,
                          w.record_elems, nthreads or default_threads())
    if rc != 0:
        raise RuntimeError(f"hs_fill_kv failed ({rc})")


def kv_records(w: Workload, layer: int, unit: int, records) -> np.ndarray:
    """uint16 [len(records)][record_elems]: regenerate individual records."""
    records = np.asarray(records, dtype=np.int64).reshape(-1)
    out = np.empty((len(records), w.record_elems), dtype=np.uint16)
    for i, r in enumerate(records):
        lib().hs_fill_kv(ctypes.c_void_p(out[i].ctypes.data), w.seed, layer, unit, 1, int(r), 1,
                         w.record_elems, 1)
    return out


def queries(w: Workload, step: int, layer: int, unit0: int = 0,
            n_units: int | None = None) -> np.ndarray:
    """uint16 (bf16 bits) [n_units][q_heads][d_qk]."""
    nu = w.units - unit0 if n_units is None else n_units
    out = np.empty((nu, w.q_heads, w.d_qk), dtype=np.uint16)
    rc = lib().hs_fill_q(ctypes.c_void_p(out.ctypes.data), w.seed ^ 0x51, step, layer, unit0, nu,
                         w.q_heads, w.d_qk)
    if rc != 0:
        raise RuntimeError(f"hs_fill_q failed ({rc})")
    return out


def normal_table() -> np.ndarray:
    p = lib().hs_normal_table()
    return np.ctypeslib.as_array(p, shape=(65536,)).copy()


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def pinned_budget_bytes() -> int:
    """Pinned host memory the inputs may use (HISPARSE_PINNED_BUDGET_GIB, default 63 GiB: a
    host that grants one process about 65 GiB of pinned memory, as measured, then fits)."""
    return int(float(os.environ.get("HISPARSE_PINNED_BUDGET_GIB", "63")) * 2**30)


def fit_pinned(w: Workload, budget: int | None = None) -> Workload:
    """The workload with as many of its layers as fit the pinned-memory budget (all other shapes
    unchanged). Per-layer work is identical, so per-layer metrics are unaffected."""
    budget = pinned_budget_bytes() if budget is None else budget
    per_layer = w.units * w.L * w.record_bytes
    n = min(w.num_layers, max(1, budget // per_layer))
    return w if n == w.num_layers else replace(w, num_layers=int(n))
