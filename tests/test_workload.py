"""The synthetic input generator: determinism and the stated selection-stream structure."""
import numpy as np
import pytest

import workload as W


def test_normal_table_is_standard_normal_quantiles():
    f = W.bf16_to_f64(W.normal_table())
    assert np.all(np.diff(f) >= 0)                 # monotone quantiles
    assert np.allclose(f, -f[::-1])                # symmetric
    assert abs(f.mean()) < 1e-6 and abs(f.std() - 1.0) < 2e-3
    from scipy.stats import norm
    p = (np.arange(65536) + 0.5) / 65536
    assert np.max(np.abs(f - norm.ppf(p)) / np.maximum(1.0, np.abs(norm.ppf(p)))) < 2 ** -8


def test_kv_is_pure_function_of_coordinates():
    w = W.workload(1)
    a = np.empty((2, 5, w.record_elems), np.uint16)
    W.fill_kv(a.ctypes.data, w, layer=0, unit0=0, n_units=2, rec0=100, n_rec=5, nthreads=3)
    b = W.kv_records(w, 0, 1, [102])
    assert (a[1, 2] == b[0]).all()
    c = np.empty((1, 1, w.record_elems), np.uint16)
    W.fill_kv(c.ctypes.data, w, layer=1, unit0=1, n_units=1, rec0=102, n_rec=1)
    assert not (c[0, 0] == b[0]).all()


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_streams_structure(n):
    w = W.workload(n)
    steps = min(w.steps, 12)
    ns = min(w.n_streams, 6)
    s = W.selection_streams(w, steps=steps, n_streams=ns)
    again = W.selection_streams(w, steps=steps, n_streams=ns)
    assert (s == again).all()
    window = set(range(w.L - w.window, w.L))
    for j in range(ns):
        for t in range(steps):
            cur = s[t, j]
            assert len(set(cur.tolist())) == w.k
            assert cur.min() >= 0 and cur.max() < w.L
            assert window <= set(cur.tolist())
            if t and w.carry:
                # exact overlap: window + carried subset
                assert len(set(cur.tolist()) & set(s[t - 1, j].tolist())) == w.window + w.carry


def test_streams_are_shuffled():
    w = W.workload(2)
    s = W.selection_streams(w, steps=2, n_streams=1)
    assert not (np.diff(s[0, 0]) > 0).all()


def test_queries_deterministic():
    w = W.workload(3)
    a = W.queries(w, 3, 2)
    b = W.queries(w, 3, 2)
    assert (a == b).all() and a.shape == (w.units, w.q_heads, w.d_qk)
    assert not (W.queries(w, 4, 2) == a).all()


def test_grow_streams_shift_window_only():
    w = W.workload(1)
    sel = W.selection_streams(w, steps=40)
    g = W.grow_streams(w, sel)
    lo = w.L - w.window
    for t in range(40):
        s, gs = sel[t, 0], g[t, 0]
        drawn = s < lo
        assert (gs[drawn] == s[drawn]).all()
        assert sorted(gs[~drawn].tolist()) == list(range(lo + t, w.L + t))
        assert len(set(gs.tolist())) == w.k


def test_correlate_layers_overlap_and_distinct():
    w = W.workload(2, num_requests=2, num_layers=3, k=64, window=8, carry=40, L=4096, B=128)
    sel = W.selection_streams(w, steps=8)
    out = W.correlate_layers(w, sel, 0.5, seed=1)
    U, lo = w.units, w.L - w.window

    def drawn(x):
        return set(x[x < lo].tolist())

    assert (out[:, :U] == sel[:, :U]).all()  # the first anchor is unchanged
    common, steady_out, steady_in = [], [], []
    for t in range(out.shape[0]):
        for s in range(out.shape[1]):
            cur, orig = out[t, s], sel[t, s]
            assert len(set(cur.tolist())) == w.k and (cur >= 0).all()  # distinct, k entries
            assert set(cur[cur >= lo].tolist()) == set(orig[orig >= lo].tolist())  # window kept
            if s >= U:
                common.append(len(drawn(cur) & drawn(out[t, s - U])))
                if t:
                    steady_out.append(len(drawn(cur) & drawn(out[t - 1, s])))
                    steady_in.append(len(drawn(orig) & drawn(sel[t - 1, s])))
    # about half of the drawn entries are shared with the previous layer (binomial spread)
    assert 0.35 * (w.k - w.window) < np.mean(common) < 0.65 * (w.k - w.window)
    # the step-to-step overlap of each layer is mostly kept
    assert np.mean(steady_out) > 0.8 * np.mean(steady_in)
    assert (W.correlate_layers(w, sel, 0.0) == sel).all()
