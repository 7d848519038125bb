"""The C ABI without a GPU: the library loads, exports every function include/hisparse.h
declares, and its pure-host validation accepts the five workloads and rejects bad descriptors."""
import ctypes
import os
import re

import pytest

import workload as W
from paper_2608_07009_amd import hisparse as hs

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "hisparse.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hisparse_[a-z_]+)\s*\(", src)))


def test_header_declares_what_binding_lists():
    assert declared_functions() == sorted(hs.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(hs.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def desc_for(w, **kw):
    d = dict(num_requests=w.num_requests, num_layers=w.num_layers,
             units_per_request=w.units_per_request, capacity=w.B, num_records=w.L, top_k=w.k,
             record_bytes=w.record_bytes, share_group=w.share_group, fetch=0, host_memory=0,
             transfer_block_bytes=0, fetch_workgroups=0)
    d.update(kw)
    return hs.CacheDesc(**d)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workload_descriptors_are_valid(cfg):
    w = W.workload(cfg)
    assert hs.hisparse_validate_desc(desc_for(w)) == hs.HISPARSE_OK
    ad = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, 0, w.scale, 0)
    assert hs.hisparse_validate_attn(w.record_bytes, w.k, ad) == hs.HISPARSE_OK
    assert hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, ad) > 0


@pytest.mark.parametrize("field,value,status", [
    ("capacity", 100, hs.HISPARSE_ERR_INVALID_ARG),          # B < k (Section 3.2 needs B >= k)
    ("top_k", 0, hs.HISPARSE_ERR_INVALID_ARG),
    ("top_k", 5000, hs.HISPARSE_ERR_INVALID_ARG),
    ("record_bytes", 1000, hs.HISPARSE_ERR_INVALID_ARG),     # not a multiple of 16
    ("num_records", 0, hs.HISPARSE_ERR_INVALID_ARG),
    ("share_group", 0, hs.HISPARSE_ERR_INVALID_ARG),
    ("num_requests", 0, hs.HISPARSE_ERR_INVALID_ARG),
    ("units_per_request", 70000, hs.HISPARSE_ERR_INVALID_ARG),
    ("fetch", 4, hs.HISPARSE_ERR_UNSUPPORTED),                # no such fetch path
    ("host_memory", 7, hs.HISPARSE_ERR_INVALID_ARG),
    ("transfer_block_bytes", 48, hs.HISPARSE_ERR_INVALID_ARG),
    ("fetch_workgroups", -1, hs.HISPARSE_ERR_INVALID_ARG),
    ("fetch_workgroups", 4097, hs.HISPARSE_ERR_INVALID_ARG),
    ("capacity", 20000, hs.HISPARSE_ERR_INVALID_ARG),        # beyond the LDS-resident maximum
])
def test_invalid_descriptors(field, value, status):
    w = W.workload(1)
    assert hs.hisparse_validate_desc(desc_for(w, **{field: value})) == status


@pytest.mark.parametrize("change,status", [
    (dict(d_qk=256), hs.HISPARSE_ERR_UNSUPPORTED),
    (dict(tokens_per_record=3), hs.HISPARSE_ERR_INVALID_ARG),
    (dict(q_heads=0), hs.HISPARSE_ERR_INVALID_ARG),
    (dict(scale=0.0), hs.HISPARSE_ERR_INVALID_ARG),
    (dict(num_splits=-1), hs.HISPARSE_ERR_INVALID_ARG),
    (dict(flags=8), hs.HISPARSE_ERR_INVALID_ARG),          # an undefined flag bit
])
def test_invalid_attention_descriptors(change, status):
    w = W.workload(2)
    d = dict(q_heads=w.q_heads, d_qk=w.d_qk, d_v=w.d_v, v_offset=w.v_offset,
             tokens_per_record=w.tokens_per_record, num_splits=0, scale=w.scale, flags=0)
    d.update(change)
    assert hs.hisparse_validate_attn(w.record_bytes, w.k, hs.AttnDesc(**d)) == status
    assert hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, hs.AttnDesc(**d)) == 0


def test_deferred_merge_flag_is_valid():
    w = W.workload(2)
    base = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, 0, w.scale, 0)
    d = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, 0, w.scale,
                    hs.HISPARSE_ATTN_DEFER_MERGE)
    assert hs.hisparse_validate_attn(w.record_bytes, w.k, d) == hs.HISPARSE_OK
    n = hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, d)
    assert n > 0 and n == hs.hisparse_decode_workspace_bytes(w.units, w.k, w.record_bytes, base)
    with pytest.raises(hs.HisparseError):  # null output / workspace: rejected on the host
        hs.hisparse_attention_merge(w.units, w.k, w.record_bytes, d, None, None, n)


def test_record_too_small_for_attention():
    ad = hs.AttnDesc(16, 576, 512, 0, 1, 0, 0.07, 0)
    assert hs.hisparse_validate_attn(512, 64, ad) == hs.HISPARSE_ERR_INVALID_ARG


def test_latent_attention_token_limit():
    """Latent attention merges at most 128 splits of at most 8192 tokens: a call with more tokens
    per unit is refused on the host (an unchecked one would index past the merge's LDS weights),
    and every accepted call's plan fits those limits."""
    R = 512 * 1152  # 512 latent tokens per record
    big = hs.AttnDesc(128, 576, 512, 0, 512, 0, 0.07, 0)
    for k in (2049, 3000, 4096):  # 2^20 + 512 .. 2^21 tokens
        assert hs.hisparse_validate_attn(R, k, big) == hs.HISPARSE_ERR_UNSUPPORTED
        assert hs.hisparse_decode_workspace_bytes(1, k, R, big) == 0
    assert hs.hisparse_validate_attn(R, 2048, big) == hs.HISPARSE_OK  # exactly 2^20 tokens
    for splits in (0, 1, 64, 200):
        d = hs.AttnDesc(128, 576, 512, 0, 512, splits, 0.07, 0)
        n = hs.hisparse_decode_workspace_bytes(1, 2048, R, d)
        # [parts][128 heads][512] fp32 partials, then [parts][128] (max, sum) pairs
        parts = n // (128 * 512 * 4 + 128 * 8)
        assert n > 0 and 1 <= parts <= 128, (splits, n)
    # token records and GQA pages are unaffected by the latent limit
    g = hs.AttnDesc(4, 128, 128, 128, 4096, 0, 0.088, 0)
    assert hs.hisparse_validate_attn(4096 * 512, 4096, g) == hs.HISPARSE_OK


def test_status_strings():
    for code, name in [(0, "HISPARSE_OK"), (-1, "HISPARSE_ERR_INVALID_ARG"),
                       (-5, "HISPARSE_ERR_BAD_SELECTION"), (-6, "HISPARSE_ERR_FULL")]:
        assert hs.hisparse_status_string(code) == name


def test_create_fails_cleanly_without_a_device_or_with_bad_args():
    w = W.workload(1)
    with pytest.raises(hs.HisparseError) as e:
        hs.hisparse_cache_create(desc_for(w, capacity=1))
    assert e.value.status == hs.HISPARSE_ERR_INVALID_ARG


def test_loads_in_a_process_that_imported_torch_first():
    """torch brings its own HIP runtime; the library must not need symbols newer than it has."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = "import torch; from paper_2608_07009_amd import hisparse as hs; hs.lib()"
    subprocess.check_call([sys.executable, "-c", code], cwd=root)


def test_entry_points_reject_a_null_handle_on_the_host():
    """Every handle-taking call validates its arguments before any GPU work (no device here)."""
    L = hs.lib()
    dummy = ctypes.c_void_p(16)  # never dereferenced: the null handle is rejected first
    r = ctypes.c_int32()
    calls = [
        lambda: L.hisparse_request_acquire(None, ctypes.byref(r)),
        lambda: L.hisparse_request_release(None, 0, None),
        lambda: L.hisparse_reset_units(None, 0, 1, None),
        lambda: L.hisparse_stage(None, 0, 1, 0, 1, 0, 1, dummy, 0, None),
        lambda: L.hisparse_speculate(None, 0, dummy, None, None),
        lambda: L.hisparse_append(None, 0, 1, dummy, dummy, dummy, None),
        lambda: L.hisparse_resolve(None, 0, dummy, dummy, None, None),
        lambda: L.hisparse_prefetch_layer(None, 0, 1, None),
        lambda: L.hisparse_fetch_turn(None, 0, dummy, 4, -1, 0, 256, None),
        lambda: L.hisparse_reset(None, None),
        # the link turns' reset checks its array and count before launching anything
        lambda: L.hisparse_link_turns_reset(None, 4, None),
        lambda: L.hisparse_link_turns_reset(dummy, 0, None),
        lambda: L.hisparse_link_turns_reset(dummy, (1 << 24) + 1, None),
    ]
    for call in calls:
        assert call() == hs.HISPARSE_ERR_INVALID_ARG


def test_largest_topk_and_capacity_are_valid():
    w = W.workload(2)
    assert hs.hisparse_validate_desc(desc_for(w, top_k=4096, capacity=16384)) == hs.HISPARSE_OK
    assert hs.hisparse_validate_desc(desc_for(w, top_k=4097, capacity=16384)) == \
        hs.HISPARSE_ERR_INVALID_ARG
    assert hs.hisparse_validate_desc(desc_for(w, top_k=4096, capacity=16385)) == \
        hs.HISPARSE_ERR_INVALID_ARG


def test_phase_timing_build_is_a_separate_library():
    """The phase-timing variant exports the same ABI; the normal library compiles none of the
    stamps and refuses to read them (no device is touched)."""
    from paper_2608_07009_amd import build as hip_build
    assert hs.lib().hisparse_debug_resolve_phases(None, 1, None) == hs.HISPARSE_ERR_UNSUPPORTED
    with pytest.raises(hs.HisparseError) as e:
        hs.hisparse_debug_resolve_phases(4)
    assert e.value.status == hs.HISPARSE_ERR_UNSUPPORTED
    assert os.path.exists(hip_build.PHASE_STAMPS_LIB_PATH), "build() makes both libraries"
    lib = ctypes.CDLL(hip_build.PHASE_STAMPS_LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    lib.hisparse_debug_resolve_phases.restype = ctypes.c_int32
    lib.hisparse_debug_resolve_phases.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
    # argument checks come before any device call
    assert lib.hisparse_debug_resolve_phases(None, 4, None) == hs.HISPARSE_ERR_INVALID_ARG


@pytest.mark.parametrize("units,splits_own,splits_beside", [(16, 8, 4), (32, 4, 2), (8, 16, 8)])
def test_beside_fetch_plan_takes_half_the_workgroups(units, splits_own, splits_beside):
    """The beside-fetch hint halves a latent-attention call's split count (so its workgroups and
    its split partials): the workspace holds [parts][128 heads][512] fp32 partials, 256-byte
    aligned, then [parts][128] (max, sum) pairs per unit."""
    w = W.workload(2)

    def parts(flags):
        d = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, 0, w.scale,
                        flags)
        n = hs.hisparse_decode_workspace_bytes(units, w.k, w.record_bytes, d)
        per_part = units * (w.q_heads * w.d_v * 4 + w.q_heads * 8)
        assert n > 0 and n % 8 == 0
        return round(n / per_part)

    assert parts(0) == splits_own
    assert parts(hs.HISPARSE_ATTN_BESIDE_FETCH) == splits_beside


@pytest.mark.parametrize("units,splits_plain,splits_carry", [(1, 32, 16), (2, 32, 16), (4, 16, 16),
                                                            (16, 8, 8)])
def test_carries_replay_plan_takes_longer_splits(units, splits_plain, splits_carry):
    """The carries-replay hint gives latent attention with one token group per workgroup (fewer
    than 16 workgroup columns) splits of at least 4 chunks of 32 tokens: for one or two units of
    128 heads at k = 2048 half the splits (and split partials); from 4 units on the plan already
    takes 4-chunk splits, and with two token groups (16 units) the hint changes nothing."""
    w = W.workload(2)

    def parts(flags):
        d = hs.AttnDesc(w.q_heads, w.d_qk, w.d_v, w.v_offset, w.tokens_per_record, 0, w.scale,
                        flags)
        n = hs.hisparse_decode_workspace_bytes(units, w.k, w.record_bytes, d)
        per_part = units * (w.q_heads * w.d_v * 4 + w.q_heads * 8)
        return round(n / per_part)

    assert parts(0) == splits_plain
    assert parts(hs.HISPARSE_ATTN_CARRIES_REPLAY) == splits_carry
    assert parts(hs.HISPARSE_ATTN_CARRIES_REPLAY | hs.HISPARSE_ATTN_DEFER_MERGE) == splits_carry
