"""A small owner of one HiSparse cache handle (create/destroy plus numpy views of host-side
state). All work is done by libhisparse.so."""
from __future__ import annotations

import numpy as np

from . import hisparse as hs


class HiSparseCache:
    def __init__(self, *, num_requests: int, num_layers: int, units_per_request: int,
                 capacity: int, num_records: int, top_k: int, record_bytes: int,
                 share_group: int = 1, fetch: int = hs.HISPARSE_FETCH_ZERO_COPY,
                 host_memory: int = hs.HISPARSE_HOST_COHERENT, transfer_block_bytes: int = 0,
                 fetch_workgroups: int = 0, device: int = 0):
        self.desc = hs.CacheDesc(num_requests, num_layers, units_per_request, capacity,
                                 num_records, top_k, record_bytes, share_group, fetch,
                                 host_memory, transfer_block_bytes, fetch_workgroups)
        self.units = num_requests * units_per_request
        self.handle = hs.hisparse_cache_create(self.desc, device)

    @classmethod
    def for_workload(cls, w, **kw) -> "HiSparseCache":
        return cls(num_requests=w.num_requests, num_layers=w.num_layers,
                   units_per_request=w.units_per_request, capacity=w.B, num_records=w.L,
                   top_k=w.k, record_bytes=w.record_bytes, share_group=w.share_group, **kw)

    def close(self) -> None:
        if self.handle:
            hs.hisparse_cache_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def L(self) -> int:
        return self.desc.num_records

    @property
    def B(self) -> int:
        return self.desc.capacity

    @property
    def k(self) -> int:
        return self.desc.top_k

    @property
    def R(self) -> int:
        return self.desc.record_bytes

    def host_pool(self, layer: int) -> tuple[int, int]:
        return hs.hisparse_host_pool(self.handle, layer)

    def host_view(self, layer: int) -> np.ndarray:
        """uint8 [units][L][R] view of a layer's pinned host pool."""
        ptr, n = self.host_pool(layer)
        return hs.host_view(ptr, n).reshape(self.units, self.L, self.R)

    def layer_cache(self, layer: int) -> tuple[int, int]:
        return hs.hisparse_layer_cache(self.handle, layer)

    def read_state(self, layer: int, page_table: bool = True) -> dict:
        U, B, L = self.units, self.B, self.L
        st = dict(slot_pos=np.empty((U, B), np.int32), slot_ts=np.empty((U, B), np.uint32),
                  order=np.empty((U, B), np.int32), clock=np.empty(U, np.uint32))
        pt = np.empty((U, L), np.int32) if page_table else None
        hs.hisparse_read_state(self.handle, layer, st["slot_pos"], st["slot_ts"], pt,
                               st["order"], st["clock"])
        if page_table:
            st["page_table"] = pt
        return st

    def read_plan(self, layer: int) -> tuple[np.ndarray, np.ndarray]:
        plan = np.empty((self.units, self.k, 2), np.int32)
        count = np.empty(self.units, np.int32)
        hs.hisparse_read_plan(self.handle, layer, plan, count)
        return plan, count

    def check_errors(self):
        return hs.hisparse_check_errors(self.handle)
