"""ctypes binding of libhisparse.so (declared in include/hisparse.h).

Argument marshalling only: every function forwards to the C ABI entry point of the same name.
Device pointers and streams are plain integers; torch tensors (anything with `data_ptr()`) and
torch streams (anything with `cuda_stream`) are accepted in their place. The library must be
built (python -m paper_2608_07009_amd.build); nothing here falls back to another
implementation when it is missing.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libhisparse.so")

HISPARSE_OK = 0
HISPARSE_ERR_INVALID_ARG = -1
HISPARSE_ERR_OOM = -2
HISPARSE_ERR_HIP = -3
HISPARSE_ERR_UNSUPPORTED = -4
HISPARSE_ERR_BAD_SELECTION = -5
HISPARSE_ERR_FULL = -6

HISPARSE_FETCH_ZERO_COPY = 0
HISPARSE_FETCH_SDMA = 1
HISPARSE_FETCH_NONE = 2
HISPARSE_FETCH_STAGED = 3

HISPARSE_ATTN_DEFER_MERGE = 1
HISPARSE_ATTN_BESIDE_FETCH = 2
HISPARSE_ATTN_CARRIES_REPLAY = 4
HISPARSE_NOALLOC_SCRATCH_BYTES = 64 << 20

HISPARSE_RESOLVE_PHASE_SLOTS = 16
HISPARSE_RESOLVE_PHASE_UNITS = 64

HISPARSE_HOST_COHERENT = 0
HISPARSE_HOST_NONCOHERENT = 1
HISPARSE_HOST_UNCACHED = 2

# Every symbol the header declares; tests check that the library exports each one.
EXPORTED = (
    "hisparse_status_string", "hisparse_validate_desc", "hisparse_validate_attn",
    "hisparse_cache_create", "hisparse_cache_destroy", "hisparse_host_pool",
    "hisparse_layer_cache", "hisparse_reset", "hisparse_resolve", "hisparse_resolve_tables",
    "hisparse_fetch", "hisparse_fetch_part", "hisparse_fetch_turn", "hisparse_link_turns_reset",
    "hisparse_fetch_units", "hisparse_fetch_group", "hisparse_prefetch_layer",
    "hisparse_prefetch_layers", "hisparse_append", "hisparse_request_acquire",
    "hisparse_request_release", "hisparse_reset_units", "hisparse_stage", "hisparse_speculate",
    "hisparse_decode_workspace_bytes", "hisparse_sparse_decode", "hisparse_sparse_decode_layers",
    "hisparse_attention_merge",
    "hisparse_sparse_decode_prefetch", "hisparse_sparse_decode_prefetch_part",
    "hisparse_attention_merge_prefetch",
    "hisparse_sparse_decode_pool", "hisparse_sparse_decode_noalloc",
    "hisparse_read_state", "hisparse_read_plan", "hisparse_check_errors",
    "hisparse_debug_resolve_phases",
)


class CacheDesc(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("units_per_request", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("num_records", ctypes.c_int64), ("top_k", ctypes.c_int32),
                ("record_bytes", ctypes.c_int32), ("share_group", ctypes.c_int32),
                ("fetch", ctypes.c_int32), ("host_memory", ctypes.c_int32),
                ("transfer_block_bytes", ctypes.c_int32), ("fetch_workgroups", ctypes.c_int32)]


class AttnDesc(ctypes.Structure):
    _fields_ = [("q_heads", ctypes.c_int32), ("d_qk", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("v_offset", ctypes.c_int32), ("tokens_per_record", ctypes.c_int32),
                ("num_splits", ctypes.c_int32), ("scale", ctypes.c_float),
                ("flags", ctypes.c_int32)]


class HisparseError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} -> {hisparse_status_string(status)} ({status})")
        self.status = status


_lib = None
_V = ctypes.c_void_p
_I32 = ctypes.c_int32


def lib() -> ctypes.CDLL:
    """Load libhisparse.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_07009_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "hisparse_status_string": (ctypes.c_char_p, [_I32]),
            "hisparse_validate_desc": (_I32, [ctypes.POINTER(CacheDesc)]),
            "hisparse_validate_attn": (_I32, [_I32, _I32, ctypes.POINTER(AttnDesc)]),
            "hisparse_cache_create": (_I32, [ctypes.POINTER(CacheDesc), _I32, ctypes.POINTER(_V)]),
            "hisparse_cache_destroy": (_I32, [_V]),
            "hisparse_host_pool": (_I32, [_V, _I32, ctypes.POINTER(_V),
                                          ctypes.POINTER(ctypes.c_size_t)]),
            "hisparse_layer_cache": (_I32, [_V, _I32, ctypes.POINTER(_V),
                                            ctypes.POINTER(ctypes.c_size_t)]),
            "hisparse_reset": (_I32, [_V, _V]),
            "hisparse_request_acquire": (_I32, [_V, ctypes.POINTER(_I32)]),
            "hisparse_request_release": (_I32, [_V, _I32, _V]),
            "hisparse_reset_units": (_I32, [_V, _I32, _I32, _V]),
            "hisparse_speculate": (_I32, [_V, _I32, _V, _V, _V]),
            "hisparse_stage": (_I32, [_V, _I32, _I32, _I32, _I32, ctypes.c_int64,
                                      ctypes.c_int64, _V, ctypes.c_int64, _V]),
            "hisparse_resolve": (_I32, [_V, _I32, _V, _V, _V, _V]),
            "hisparse_resolve_tables": (_I32, [_V, _I32, _V, _V, _V, _V]),
            "hisparse_fetch": (_I32, [_V, _I32, _V]),
            "hisparse_fetch_part": (_I32, [_V, _I32, _I32, _I32, _V]),
            "hisparse_fetch_turn": (_I32, [_V, _I32, _V, _I32, _I32, _I32, _I32, _V]),
            "hisparse_link_turns_reset": (_I32, [_V, _I32, _V]),
            "hisparse_fetch_units": (_I32, [_V, _I32, _I32, _I32, _V]),
            "hisparse_fetch_group": (_I32, [_V, _I32, _I32, _V]),
            "hisparse_prefetch_layer": (_I32, [_V, _I32, _I32, _V]),
            "hisparse_prefetch_layers": (_I32, [_V, _I32, _I32, _I32, _V]),
            "hisparse_append": (_I32, [_V, _I32, _I32, _V, _V, _V, _V]),
            "hisparse_decode_workspace_bytes": (ctypes.c_size_t, [_I32, _I32, _I32,
                                                                  ctypes.POINTER(AttnDesc)]),
            "hisparse_sparse_decode": (_I32, [_V, _I32, _V, _V, _V, ctypes.POINTER(AttnDesc), _V,
                                              ctypes.c_size_t, _V]),
            "hisparse_attention_merge": (_I32, [_I32, _I32, _I32, ctypes.POINTER(AttnDesc), _V,
                                                _V, ctypes.c_size_t, _V]),
            "hisparse_sparse_decode_layers": (_I32, [_V, _I32, _I32, _V, _V, _V,
                                                     ctypes.POINTER(AttnDesc), _V,
                                                     ctypes.c_size_t, _V]),
            "hisparse_sparse_decode_prefetch": (_I32, [_V, _I32, _V, _V, _V,
                                                       ctypes.POINTER(AttnDesc), _V,
                                                       ctypes.c_size_t, _I32, _I32, _I32, _V]),
            "hisparse_sparse_decode_noalloc": (_I32, [_V, _I32, _V, _V, _V,
                                                      ctypes.POINTER(AttnDesc), _V]),
            "hisparse_sparse_decode_prefetch_part": (_I32, [_V, _I32, _V, _V, _V,
                                                            ctypes.POINTER(AttnDesc), _V,
                                                            ctypes.c_size_t, _I32, _I32, _I32,
                                                            _I32, _I32, _V]),
            "hisparse_attention_merge_prefetch": (_I32, [_V, ctypes.POINTER(AttnDesc), _V, _V,
                                                         ctypes.c_size_t, _I32, _I32, _I32,
                                                         _I32, _I32, _V]),
            "hisparse_sparse_decode_pool": (_I32, [_V, ctypes.c_int64, _I32, _I32, _I32, _V, _V,
                                                   _V, ctypes.POINTER(AttnDesc), _V,
                                                   ctypes.c_size_t, _V]),
            "hisparse_read_state": (_I32, [_V, _I32, _V, _V, _V, _V, _V]),
            "hisparse_read_plan": (_I32, [_V, _I32, _V, _V]),
            "hisparse_check_errors": (_I32, [_V, _V]),
            "hisparse_debug_resolve_phases": (_I32, [_V, _I32, ctypes.POINTER(ctypes.c_int64)]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p(x) -> int | None:
    """Raw address of a pointer-like argument (int, torch tensor, numpy array or None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)!r}")


def _s(stream) -> int | None:
    if stream is None or isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(fn: str, status: int) -> None:
    if status != HISPARSE_OK:
        raise HisparseError(fn, status)


def hisparse_status_string(status: int) -> str:
    return lib().hisparse_status_string(status).decode()


def hisparse_validate_desc(desc: CacheDesc) -> int:
    return lib().hisparse_validate_desc(ctypes.byref(desc))


def hisparse_validate_attn(record_bytes: int, top_k: int, attn: AttnDesc) -> int:
    return lib().hisparse_validate_attn(record_bytes, top_k, ctypes.byref(attn))


def hisparse_cache_create(desc: CacheDesc, device: int = 0) -> int:
    h = _V()
    _check("hisparse_cache_create", lib().hisparse_cache_create(ctypes.byref(desc), device,
                                                               ctypes.byref(h)))
    return h.value


def hisparse_cache_destroy(cache: int) -> None:
    _check("hisparse_cache_destroy", lib().hisparse_cache_destroy(cache))


def hisparse_host_pool(cache: int, layer: int) -> tuple[int, int]:
    p, n = _V(), ctypes.c_size_t()
    _check("hisparse_host_pool", lib().hisparse_host_pool(cache, layer, ctypes.byref(p),
                                                         ctypes.byref(n)))
    return p.value, n.value


def hisparse_layer_cache(cache: int, layer: int) -> tuple[int, int]:
    p, n = _V(), ctypes.c_size_t()
    _check("hisparse_layer_cache", lib().hisparse_layer_cache(cache, layer, ctypes.byref(p),
                                                             ctypes.byref(n)))
    return p.value, n.value


def hisparse_reset(cache: int, stream=None) -> None:
    _check("hisparse_reset", lib().hisparse_reset(cache, _s(stream)))


def hisparse_request_acquire(cache: int) -> int:
    r = _I32()
    _check("hisparse_request_acquire", lib().hisparse_request_acquire(cache, ctypes.byref(r)))
    return r.value


def hisparse_request_release(cache: int, request: int, stream=None) -> None:
    _check("hisparse_request_release", lib().hisparse_request_release(cache, request,
                                                                     _s(stream)))


def hisparse_reset_units(cache: int, first_unit: int, num_units: int, stream=None) -> None:
    _check("hisparse_reset_units", lib().hisparse_reset_units(cache, first_unit, num_units,
                                                             _s(stream)))


def hisparse_stage(cache: int, first_layer: int, num_layers: int, first_unit: int,
                   num_units: int, first_record: int, num_records: int, d_src,
                   src_layer_stride: int = 0, stream=None) -> None:
    _check("hisparse_stage", lib().hisparse_stage(cache, first_layer, num_layers, first_unit,
                                                 num_units, first_record, num_records,
                                                 _p(d_src), src_layer_stride, _s(stream)))


def hisparse_speculate(cache: int, layer: int, d_hint, d_counts=None, stream=None) -> None:
    _check("hisparse_speculate", lib().hisparse_speculate(cache, layer, _p(d_hint), _p(d_counts),
                                                         _s(stream)))


def hisparse_resolve(cache: int, layer: int, d_sel, d_slots, d_counts=None, stream=None) -> None:
    _check("hisparse_resolve", lib().hisparse_resolve(cache, layer, _p(d_sel), _p(d_slots),
                                                     _p(d_counts), _s(stream)))


def hisparse_resolve_tables(cache: int, layer: int, d_sel, d_slots, d_counts=None,
                            stream=None) -> None:
    _check("hisparse_resolve_tables",
           lib().hisparse_resolve_tables(cache, layer, _p(d_sel), _p(d_slots), _p(d_counts),
                                         _s(stream)))


def hisparse_fetch(cache: int, layer: int, stream=None) -> None:
    _check("hisparse_fetch", lib().hisparse_fetch(cache, layer, _s(stream)))


def hisparse_fetch_part(cache: int, layer: int, part_begin: int, part_end: int,
                        stream=None) -> None:
    _check("hisparse_fetch_part",
           lib().hisparse_fetch_part(cache, layer, part_begin, part_end, _s(stream)))


def hisparse_fetch_turn(cache: int, layer: int, d_turns, n_turns: int, wait_turn: int,
                        signal_turn: int, signal_share: int = 256, stream=None) -> None:
    _check("hisparse_fetch_turn",
           lib().hisparse_fetch_turn(cache, layer, _p(d_turns), n_turns, wait_turn, signal_turn,
                                     signal_share, _s(stream)))


def hisparse_link_turns_reset(d_turns, n_turns: int, stream=None) -> None:
    _check("hisparse_link_turns_reset",
           lib().hisparse_link_turns_reset(_p(d_turns), n_turns, _s(stream)))


def hisparse_fetch_units(cache: int, layer: int, unit_begin: int, unit_count: int,
                         stream=None) -> None:
    _check("hisparse_fetch_units",
           lib().hisparse_fetch_units(cache, layer, unit_begin, unit_count, _s(stream)))


def hisparse_fetch_group(cache: int, anchor_layer: int, num_layers: int, stream=None) -> None:
    _check("hisparse_fetch_group",
           lib().hisparse_fetch_group(cache, anchor_layer, num_layers, _s(stream)))


def hisparse_prefetch_layer(cache: int, anchor_layer: int, shared_layer: int,
                            stream=None) -> None:
    _check("hisparse_prefetch_layer",
           lib().hisparse_prefetch_layer(cache, anchor_layer, shared_layer, _s(stream)))


def hisparse_append(cache: int, first_layer: int, num_layers: int, pos, records, slots,
                    stream=None) -> None:
    _check("hisparse_append",
           lib().hisparse_append(cache, first_layer, num_layers, _p(pos), _p(records), _p(slots),
                                 _s(stream)))


def hisparse_prefetch_layers(cache: int, anchor_layer: int, first_shared: int, num_layers: int,
                             stream=None) -> None:
    _check("hisparse_prefetch_layers",
           lib().hisparse_prefetch_layers(cache, anchor_layer, first_shared, num_layers,
                                          _s(stream)))


def hisparse_decode_workspace_bytes(units: int, top_k: int, record_bytes: int,
                                    attn: AttnDesc) -> int:
    return lib().hisparse_decode_workspace_bytes(units, top_k, record_bytes, ctypes.byref(attn))


def hisparse_sparse_decode(cache: int, layer: int, d_q, d_slots, d_out, attn: AttnDesc,
                           d_workspace, workspace_bytes: int, stream=None) -> None:
    _check("hisparse_sparse_decode",
           lib().hisparse_sparse_decode(cache, layer, _p(d_q), _p(d_slots), _p(d_out),
                                        ctypes.byref(attn), _p(d_workspace), workspace_bytes,
                                        _s(stream)))


def hisparse_sparse_decode_noalloc(cache: int, layer: int, d_q, d_slots, d_out, attn: AttnDesc,
                                   stream=None) -> None:
    _check("hisparse_sparse_decode_noalloc",
           lib().hisparse_sparse_decode_noalloc(cache, layer, _p(d_q), _p(d_slots), _p(d_out),
                                                ctypes.byref(attn), _s(stream)))


def hisparse_sparse_decode_prefetch_part(cache: int, layer: int, d_q, d_slots, d_out,
                                         attn: AttnDesc, d_workspace, workspace_bytes: int,
                                         anchor_layer: int, first_shared: int, num_shared: int,
                                         part_begin: int, part_end: int, stream=None) -> None:
    _check("hisparse_sparse_decode_prefetch_part",
           lib().hisparse_sparse_decode_prefetch_part(
               cache, layer, _p(d_q), _p(d_slots), _p(d_out), ctypes.byref(attn),
               _p(d_workspace), workspace_bytes, anchor_layer, first_shared, num_shared,
               part_begin, part_end, _s(stream)))


def hisparse_attention_merge_prefetch(cache: int, attn: AttnDesc, d_out, d_workspace,
                                      workspace_bytes: int, anchor_layer: int, first_shared: int,
                                      num_shared: int, part_begin: int, part_end: int,
                                      stream=None) -> None:
    _check("hisparse_attention_merge_prefetch",
           lib().hisparse_attention_merge_prefetch(
               cache, ctypes.byref(attn), _p(d_out), _p(d_workspace), workspace_bytes,
               anchor_layer, first_shared, num_shared, part_begin, part_end, _s(stream)))


def hisparse_attention_merge(units: int, top_k: int, record_bytes: int, attn: AttnDesc, d_out,
                             d_workspace, workspace_bytes: int, stream=None) -> None:
    _check("hisparse_attention_merge",
           lib().hisparse_attention_merge(units, top_k, record_bytes, ctypes.byref(attn),
                                          _p(d_out), _p(d_workspace), workspace_bytes,
                                          _s(stream)))


def hisparse_sparse_decode_layers(cache: int, first_layer: int, num_layers: int, q, slots, out,
                                  attn: AttnDesc, workspace, workspace_bytes: int,
                                  stream=None) -> None:
    _check("hisparse_sparse_decode_layers",
           lib().hisparse_sparse_decode_layers(cache, first_layer, num_layers, _p(q), _p(slots),
                                               _p(out), ctypes.byref(attn), _p(workspace),
                                               workspace_bytes, _s(stream)))


def hisparse_sparse_decode_prefetch(cache: int, layer: int, q, slots, out, attn: AttnDesc,
                                    workspace, workspace_bytes: int, anchor_layer: int,
                                    first_shared: int, num_shared: int, stream=None) -> None:
    _check("hisparse_sparse_decode_prefetch",
           lib().hisparse_sparse_decode_prefetch(cache, layer, _p(q), _p(slots), _p(out),
                                                 ctypes.byref(attn), _p(workspace),
                                                 workspace_bytes, anchor_layer, first_shared,
                                                 num_shared, _s(stream)))


def hisparse_sparse_decode_pool(d_pool, records_per_unit: int, record_bytes: int, units: int,
                                top_k: int, d_q, d_idx, d_out, attn: AttnDesc, d_workspace,
                                workspace_bytes: int, stream=None) -> None:
    _check("hisparse_sparse_decode_pool",
           lib().hisparse_sparse_decode_pool(_p(d_pool), records_per_unit, record_bytes, units,
                                             top_k, _p(d_q), _p(d_idx), _p(d_out),
                                             ctypes.byref(attn), _p(d_workspace),
                                             workspace_bytes, _s(stream)))


def hisparse_read_state(cache: int, layer: int, slot_pos=None, slot_ts=None, page_table=None,
                        order=None, clock=None) -> None:
    _check("hisparse_read_state",
           lib().hisparse_read_state(cache, layer, _p(slot_pos), _p(slot_ts), _p(page_table),
                                     _p(order), _p(clock)))


def hisparse_read_plan(cache: int, layer: int, plan=None, count=None) -> None:
    _check("hisparse_read_plan", lib().hisparse_read_plan(cache, layer, _p(plan), _p(count)))


def hisparse_check_errors(cache: int) -> tuple[int, tuple[int, int, int]]:
    info = (ctypes.c_int32 * 3)()
    st = lib().hisparse_check_errors(cache, ctypes.cast(info, _V))
    if st not in (HISPARSE_OK, HISPARSE_ERR_BAD_SELECTION):
        raise HisparseError("hisparse_check_errors", st)
    return st, (info[0], info[1], info[2])


def hisparse_debug_resolve_phases(max_units: int) -> tuple[np.ndarray, int]:
    """(uint64 [units][HISPARSE_RESOLVE_PHASE_SLOTS] stamps of the last resolve launch, clock
    ticks per second); raises HisparseError (UNSUPPORTED) unless the library is a phase-timing
    build."""
    n = max(1, min(max_units, HISPARSE_RESOLVE_PHASE_UNITS))
    out = np.zeros((n, HISPARSE_RESOLVE_PHASE_SLOTS), dtype=np.uint64)
    rate = ctypes.c_int64(0)
    _check("hisparse_debug_resolve_phases",
           lib().hisparse_debug_resolve_phases(out.ctypes.data, n, ctypes.byref(rate)))
    return out, rate.value


def host_view(ptr: int, nbytes: int, dtype=np.uint8) -> np.ndarray:
    """Zero-copy numpy view of host memory (e.g. a layer's pinned host pool)."""
    buf = (ctypes.c_uint8 * nbytes).from_address(ptr)
    return np.frombuffer(buf, dtype=dtype)
