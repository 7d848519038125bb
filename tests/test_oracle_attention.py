"""Pins for the oracle's float64 sparse decode attention (CPU only).

Section 3.1 "Exact sparse-attention outputs": placement must not change the attention over the
selected set. The oracle is pinned against:
  * torch's scaled_dot_product_attention in float64 on explicitly gathered keys/values (an
    independent library routine for softmax attention);
  * closed forms: a single token returns its value exactly; identical keys give the mean of
    the values; a dominant score returns that token's value;
  * placement independence: the GPU-cache image addressed through slots gives the very same
    doubles as the full pool addressed through positions;
  * padding entries are ignored.
"""
import numpy as np
import pytest
import torch

import oracle
import workload


def bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def to_f64(bits):
    return workload.bf16_to_f64(bits)


def sdpa_ref(q64, k64, v64, scale):
    q = torch.from_numpy(q64)[:, None, :]  # [H, 1, d]
    k = torch.from_numpy(k64)[None].expand(q.shape[0], -1, -1)
    v = torch.from_numpy(v64)[None].expand(q.shape[0], -1, -1)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale)
    return o[:, 0, :].numpy()


@pytest.mark.parametrize("kind", ["mla", "gqa"])
def test_matches_library_sdpa(kind):
    rng = np.random.default_rng(11)
    if kind == "mla":
        H, dqk, dv, voff, te, tpr, scale = 8, 576, 512, 0, 576, 1, 1 / np.sqrt(192)
    else:
        H, dqk, dv, voff, te, tpr, scale = 4, 128, 128, 128, 256, 4, 1 / np.sqrt(128)
    n_rec, k = 60, 17
    pool = bf16_bits(rng.standard_normal((n_rec, tpr * te)))
    q = bf16_bits(rng.standard_normal((H, dqk)))
    idx = rng.choice(n_rec, size=k, replace=False).astype(np.int32)
    out = oracle.sparse_decode(q, pool, idx, d_qk=dqk, d_v=dv, v_off=voff, token_elems=te,
                               tokens_per_record=tpr, scale=scale)
    toks = to_f64(pool[idx].reshape(k * tpr, te))
    ref = sdpa_ref(to_f64(q), toks[:, :dqk].copy(), toks[:, voff:voff + dv].copy(), scale)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_single_token_returns_value_exactly():
    rng = np.random.default_rng(12)
    pool = bf16_bits(rng.standard_normal((5, 576)))
    q = bf16_bits(rng.standard_normal((3, 576)))
    out = oracle.sparse_decode(q, pool, [3], d_qk=576, d_v=512, v_off=0, token_elems=576,
                               tokens_per_record=1, scale=0.1)
    assert (out == to_f64(pool[3, :512])[None]).all()


def test_identical_keys_give_mean_value():
    rng = np.random.default_rng(13)
    te = 256
    keys = bf16_bits(rng.standard_normal(128))
    pool = bf16_bits(rng.standard_normal((10, te)))
    pool[:, :128] = keys
    q = bf16_bits(rng.standard_normal((2, 128)))
    out = oracle.sparse_decode(q, pool, np.arange(10), d_qk=128, d_v=128, v_off=128,
                               token_elems=te, tokens_per_record=1, scale=0.3)
    np.testing.assert_allclose(out, np.broadcast_to(to_f64(pool[:, 128:]).mean(0), out.shape),
                               rtol=1e-13, atol=1e-14)


def test_dominant_score_and_no_overflow():
    rng = np.random.default_rng(14)
    pool = bf16_bits(rng.standard_normal((6, 64)))
    q = pool[4:5, :32].copy()  # q == key of record 4
    out = oracle.sparse_decode(q, pool, np.arange(6), d_qk=32, d_v=32, v_off=32, token_elems=64,
                               tokens_per_record=1, scale=1e4)
    assert np.isfinite(out).all()
    np.testing.assert_allclose(out[0], to_f64(pool[4, 32:]), atol=1e-12)


def test_cache_image_equals_full_pool_bitwise():
    # The same records, placed in arbitrary slots, give bit-identical float64 outputs.
    rng = np.random.default_rng(15)
    L, B, k = 200, 48, 24
    pool = bf16_bits(rng.standard_normal((L, 576)))
    q = bf16_bits(rng.standard_normal((4, 576)))
    c = oracle.OracleCache(1, L, B, k)
    cache = np.zeros((B, 576), dtype=np.uint16)
    for t in range(6):
        sel = rng.choice(L, size=k, replace=False).astype(np.int32)
        rc, slots, counts, pp, ps = c.resolve_unit(0, sel)
        oracle.apply_plan(pool, cache, pp, ps)
        kw = dict(d_qk=576, d_v=512, v_off=0, token_elems=576, tokens_per_record=1, scale=0.07)
        a = oracle.sparse_decode(q, pool, sel, **kw)
        b = oracle.sparse_decode(q, cache, slots, **kw)
        assert a.tobytes() == b.tobytes()


def test_padding_ignored_and_empty_is_zero():
    rng = np.random.default_rng(16)
    pool = bf16_bits(rng.standard_normal((9, 256)))
    q = bf16_bits(rng.standard_normal((2, 128)))
    kw = dict(d_qk=128, d_v=128, v_off=128, token_elems=256, tokens_per_record=1, scale=0.2)
    a = oracle.sparse_decode(q, pool, [5, -1, 2, -1, 7], **kw)
    b = oracle.sparse_decode(q, pool, [5, 2, 7], **kw)
    assert a.tobytes() == b.tobytes()
    z = oracle.sparse_decode(q, pool, [-1, -1], **kw)
    assert (z == 0).all()
