"""HiSparse CPU oracle (test infrastructure only).

ctypes access to `hisparse_oracle.c`, the plain, slow, float64 reference of the resolve step
(Section 3.2 data model and replacement policy, Section 3.4 phases) and of sparse decode
attention (Section 3.1 exactness invariant). Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product library never does.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_DIR = os.path.join(_HERE, "lib")
_LIB_PATH = os.path.join(_LIB_DIR, "libhisparse_oracle.so")
_SRC = os.path.join(_HERE, "hisparse_oracle.c")

OK = 0
BAD_SELECTION = -5


def build(force: bool = True, path: str | None = None, extra_flags=()) -> str:
    """Compile the oracle with gcc (no HIP) into oracle/lib/libhisparse_oracle.so, or into
    `path` with extra compiler flags (e.g. a sanitizer build)."""
    out = path or _LIB_PATH
    os.makedirs(os.path.dirname(out), exist_ok=True)
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
                               "-fno-fast-math", "-ffp-contract=off", *extra_flags, _SRC,
                               "-o", tmp, "-lm"])
        os.replace(tmp, out)
    return out


_lib = None
_P = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("HISPARSE_ORACLE_LIB") or _LIB_PATH  # another build, e.g. sanitized
        if not os.path.exists(path):
            raise RuntimeError("oracle not built: run __graft_entry__.build()")
        L = ctypes.CDLL(path)
        L.oracle_resolve.restype = ctypes.c_int
        L.oracle_resolve.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32] + [_P] * 9
        L.oracle_resolve_units.restype = ctypes.c_int
        L.oracle_resolve_units.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32,
                                           ctypes.c_int32] + [_P] * 9
        L.oracle_apply_plan.restype = None
        L.oracle_apply_plan.argtypes = [_P, _P, ctypes.c_int32, _P, _P, ctypes.c_int32]
        L.oracle_sparse_decode.restype = ctypes.c_int
        L.oracle_sparse_decode.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, _P,
                                           ctypes.c_int32, ctypes.c_double, _P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


class OracleCache:
    """Resolve state of `n_units` independent caches with B slots over L records each."""

    def __init__(self, n_units: int, L: int, B: int, k: int):
        self.n_units, self.L, self.B, self.k = n_units, L, B, k
        self.pt = np.full((n_units, L), -1, dtype=np.int32)
        self.slot_pos = np.full((n_units, B), -1, dtype=np.int32)
        self.slot_ts = np.zeros((n_units, B), dtype=np.uint32)
        self.clock = np.zeros(n_units, dtype=np.uint32)

    def resolve(self, sel: np.ndarray):
        """sel int32 [n_units][k] -> (slots [n_units][k], counts [n_units][2],
        plan_pos [n_units][k], plan_slot [n_units][k], n_bad)."""
        sel = np.ascontiguousarray(sel, dtype=np.int32).reshape(self.n_units, self.k)
        slots = np.empty_like(sel)
        counts = np.empty((self.n_units, 2), dtype=np.int32)
        plan_pos = np.full_like(sel, -1)
        plan_slot = np.full_like(sel, -1)
        rc = lib().oracle_resolve_units(self.n_units, self.L, self.B, self.k, _ptr(self.pt),
                                        _ptr(self.slot_pos), _ptr(self.slot_ts), _ptr(self.clock),
                                        _ptr(sel), _ptr(slots), _ptr(counts), _ptr(plan_pos),
                                        _ptr(plan_slot))
        if rc < 0:
            raise RuntimeError(f"oracle_resolve_units failed ({rc})")
        return slots, counts, plan_pos, plan_slot, rc

    def resolve_unit(self, u: int, sel: np.ndarray):
        """One unit; returns (rc, slots, counts, plan_pos[:m], plan_slot[:m])."""
        sel = np.ascontiguousarray(sel, dtype=np.int32).reshape(self.k)
        slots = np.empty_like(sel)
        counts = np.zeros(2, dtype=np.int32)
        plan_pos = np.full_like(sel, -1)
        plan_slot = np.full_like(sel, -1)
        pt = self.pt[u]
        sp = self.slot_pos[u]
        ts = self.slot_ts[u]
        clk = self.clock[u:u + 1]
        rc = lib().oracle_resolve(self.L, self.B, self.k, _ptr(pt), _ptr(sp), _ptr(ts), _ptr(clk),
                                  _ptr(sel), _ptr(slots), _ptr(counts), _ptr(plan_pos),
                                  _ptr(plan_slot))
        if rc not in (OK, BAD_SELECTION):
            raise RuntimeError(f"oracle_resolve failed ({rc})")
        m = int(counts[1])
        return rc, slots, counts, plan_pos[:m].copy(), plan_slot[:m].copy()


    def reset_unit(self, u: int) -> None:
        """Admission of a new request into unit u (Section 3.3 (2)): the unit's cache starts
        cold, exactly as at creation; the other units are untouched."""
        self.pt[u] = -1
        self.slot_pos[u] = -1
        self.slot_ts[u] = 0
        self.clock[u] = 0

    def admit_unit(self, u: int, pos: int):
        """Write-through admission of a newly generated record at position `pos` (Section 3.3
        (4)), read as a one-entry resolve event of the unit: the clock advances, a resident
        position is refreshed, otherwise the least-recent slot by (timestamp, slot) takes it
        with the event's miss stamp. Returns (rc, slot, was_hit)."""
        sel = np.array([pos], dtype=np.int32)
        slots = np.empty(1, dtype=np.int32)
        counts = np.zeros(2, dtype=np.int32)
        plan_pos = np.full(1, -1, dtype=np.int32)
        plan_slot = np.full(1, -1, dtype=np.int32)
        rc = lib().oracle_resolve(self.L, self.B, 1, _ptr(self.pt[u]), _ptr(self.slot_pos[u]),
                                  _ptr(self.slot_ts[u]), _ptr(self.clock[u:u + 1]), _ptr(sel),
                                  _ptr(slots), _ptr(counts), _ptr(plan_pos), _ptr(plan_slot))
        if rc not in (OK, BAD_SELECTION):
            raise RuntimeError(f"oracle_resolve failed ({rc})")
        return rc, int(slots[0]), bool(counts[0])


def apply_plan(host_unit: np.ndarray, cache_unit: np.ndarray, plan_pos, plan_slot) -> None:
    """cache_unit[slot] <- host_unit[pos]; both uint8/uint16 arrays [records][...]."""
    plan_pos = np.ascontiguousarray(plan_pos, dtype=np.int32)
    plan_slot = np.ascontiguousarray(plan_slot, dtype=np.int32)
    R = host_unit[0].nbytes
    assert cache_unit[0].nbytes == R and host_unit.flags.c_contiguous and cache_unit.flags.c_contiguous
    lib().oracle_apply_plan(_ptr(host_unit), _ptr(cache_unit), R, _ptr(plan_pos), _ptr(plan_slot),
                            len(plan_pos))


def sparse_decode(q: np.ndarray, pool: np.ndarray, idx, *, d_qk: int, d_v: int, v_off: int,
                  token_elems: int, tokens_per_record: int, scale: float) -> np.ndarray:
    """float64 [H][d_v] attention of q (uint16 bf16 bits [H][d_qk]) over the records of `pool`
    (uint16 [records][tokens_per_record*token_elems]) addressed by idx (-1 = padding)."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    pool = np.ascontiguousarray(pool, dtype=np.uint16)
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(-1)
    assert pool.shape[-1] == tokens_per_record * token_elems
    assert np.all(idx < pool.shape[0])
    H = q.shape[0]
    out = np.empty((H, d_v), dtype=np.float64)
    rc = lib().oracle_sparse_decode(_ptr(q), H, d_qk, d_v, v_off, token_elems, tokens_per_record,
                                    _ptr(pool), _ptr(idx), len(idx), float(scale), _ptr(out))
    if rc != OK:
        raise RuntimeError(f"oracle_sparse_decode failed ({rc})")
    return out
