"""The seeded input generators: shapes, value structure, determinism, prefixes."""
import numpy as np
import pytest

from paper_1801_01554_amd import workloads as wl
from paper_1801_01554_amd.metrics import num_weights


def test_named_workload_table():
    assert wl.ORDER == ["nettalk-80-b1024", "nettalk-120-b512", "nettalk-120-b16",
                        "wide-1024-4096-1024", "deep-512-2048x3-64"]
    assert num_weights(wl.SPECS["nettalk-120-b512"].sizes) == 27626
    assert num_weights(wl.SPECS["wide-1024-4096-1024"].sizes) == 8393728
    assert num_weights(wl.SPECS["deep-512-2048x3-64"].sizes) == 9574464


def test_onehot_window_structure():
    w = wl.make("nettalk-120-b512", n_patterns=2000)
    a = w.active
    assert a.shape == (2000, 7) and a.dtype == np.int32
    pos = a // 29
    assert np.all(pos == np.arange(7)[None, :])          # one active symbol per position
    assert a.min() >= 0 and a.max() < 203
    x = w.dense_inputs()
    assert x.shape == (2000, 203) and np.all(x.sum(1) == 7)
    sym_counts = np.bincount((a % 29).ravel(), minlength=29)
    assert sym_counts.min() > 0.7 * sym_counts.mean()    # uniform symbols
    t = w.targets
    assert set(np.unique(t)) == {np.float32(0.1), np.float32(0.9)}
    assert abs(np.mean(t == np.float32(0.9)) - 0.15) < 0.01


def test_dense_inputs_and_init_ranges():
    w = wl.make("wide-1024-4096-1024", n_patterns=64)
    assert w.inputs.shape == (64, 1024) and w.inputs.dtype == np.float32
    assert w.inputs.min() >= -1 and w.inputs.max() <= 1
    assert w.weights.size == 8393728
    W0 = w.weights[:1025 * 4096]
    assert np.abs(W0).max() <= 1 / np.sqrt(1024)
    d = wl.make("deep-512-2048x3-64", n_patterns=64)
    assert abs(d.inputs.std() - 1) < 0.05
    assert abs(np.mean(d.targets == np.float32(0.9)) - 0.5) < 0.05


@pytest.mark.parametrize("name", ["nettalk-80-b1024", "wide-1024-4096-1024"])
def test_prefix_and_determinism(name):
    a = wl.make(name, n_patterns=300)
    b = wl.make(name, n_patterns=40)
    c = wl.make(name, n_patterns=300)
    if a.inputs is not None:
        np.testing.assert_array_equal(a.inputs[:40], b.inputs)
        np.testing.assert_array_equal(a.inputs, c.inputs)
    else:
        np.testing.assert_array_equal(a.active[:40], b.active)
    np.testing.assert_array_equal(a.targets[:40], b.targets)
    np.testing.assert_array_equal(a.weights, b.weights)


def test_chunked_draw_equals_single_draw(monkeypatch):
    full = wl.draw_inputs("normal", 9, 100, 7)[0]
    monkeypatch.setattr(wl, "CHUNK_ROWS", 13)
    np.testing.assert_array_equal(wl.draw_inputs("normal", 9, 100, 7)[0], full)


def test_small_batch_case_shares_data_with_b512():
    a = wl.make("nettalk-120-b512", n_patterns=100)
    b = wl.make("nettalk-120-b16", n_patterns=100)
    np.testing.assert_array_equal(a.active, b.active)
    np.testing.assert_array_equal(a.weights, b.weights)


def test_custom_onehot_indices_distinct():
    w = wl.make_custom((50, 6, 3), 40, seed=2, onehot=True)
    for row in w.active:
        assert len(set(row.tolist())) == row.size


# --------------------------------------------------------------------------- sequences
@pytest.mark.parametrize("name", list(wl.SEQ_SPECS))
def test_sequence_layout(name):
    w = wl.make_sequences(name)
    s = w.spec
    T, S = s.n_steps, s.n_streams
    assert w.inputs.shape == (T, S, s.n_ext) and w.targets.shape == (T, S, s.n_out)
    assert w.cont.shape == w.mask.shape == (T, S)
    assert w.weights.size == wl.num_weights(s.sizes)
    for st in range(S):
        m, c = w.mask[:, st], w.cont[:, st]
        end = int(m.sum())
        assert np.all(m[:end] == 1) and np.all(m[end:] == 0)          # padding only after the last sequence
        assert np.all(c[end:] == 0) and (end == 0 or c[0] == 0)
        starts = [0] + [t for t in range(1, end) if c[t] == 0] + [end]
        lens = np.diff(starts)
        assert np.all(lens >= s.len_min) and np.all(lens <= s.len_max)
        assert T - end < s.len_max                                     # the next sequence did not fit
    # one class per frame: exactly one 0.9 target
    assert np.all(np.sum(w.targets == np.float32(0.9), axis=2) == 1)
    w2 = wl.make_sequences(name)
    np.testing.assert_array_equal(w.inputs, w2.inputs)
    np.testing.assert_array_equal(w.cont, w2.cont)
