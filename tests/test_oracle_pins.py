"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these tests retypes the oracle's formulas.  Each pins the oracle to
something else:

* the forward pass to scikit-learn's logistic model (a library routine): a
  one-layer sigmoid net IS logistic regression, and a deeper net is the
  composition of such layers;
* the summed weight change to the negative gradient of half the summed
  squared error, by central differences of the (pinned) forward pass;
* the update rule to invariants and closed forms (zero weights, lr = 0,
  linearity in lr, two consecutive batches);
* the connection count to the paper's NETtalk figure (section 6.3) and the
  MCPS-to-flops factor to the paper's 4.23 (section 7.2).

A plausible mistake anywhere in the oracle (a dropped bias term, a wrong sign
or index, a transposed operand, a mean instead of a sum, a missing derivative
factor) fails at least one of these.
"""
import numpy as np
import pytest
from sklearn.linear_model import LogisticRegression

import oracle
from paper_1801_01554_amd import workloads as wl


def _logistic_layer(x, W):
    """Applies one sigmoid layer using scikit-learn's logistic model, one output unit at a time.

    W is (n_in + 1) x n_out with the bias in the last row.
    """
    n_in, n_out = W.shape[0] - 1, W.shape[1]
    out = np.empty((x.shape[0], n_out))
    for j in range(n_out):
        m = LogisticRegression()
        m.classes_ = np.array([0, 1])
        m.coef_ = W[:n_in, j][None, :].astype(np.float64)
        m.intercept_ = np.array([W[n_in, j]], dtype=np.float64)
        out[:, j] = m.predict_proba(x.astype(np.float64))[:, 1]
    return out


def _net(sizes, w, storage=64):
    n = oracle.OracleNet(sizes, storage)
    n.set_weights(w)
    return n


def _rand_case(sizes, n, seed, scale=1.0):
    g = np.random.default_rng(seed)
    x = g.uniform(-1, 1, (n, sizes[0])).astype(np.float32)
    t = np.where(g.random((n, sizes[-1])) < 0.5, 0.9, 0.1).astype(np.float32)
    w = (g.uniform(-scale, scale, wl.num_weights(sizes))).astype(np.float32).astype(np.float64)
    return x, t, w


# --------------------------------------------------------------------------- counting
def test_connection_count_matches_nettalk():
    # Section 6.3: 203 inputs + true unit, 60 hidden, 26 outputs -> 13,826 connections.
    assert wl.num_weights((203, 60, 26)) == 13826
    assert oracle.OracleNet((203, 60, 26)).n_weights == 13826


def test_flops_per_connection_factor_matches_paper():
    # Section 7.2: MFLOPS = MCPS * (4 + 2 (W - W_i) / W) = MCPS * 4.23 for NETtalk.
    from paper_1801_01554_amd.metrics import paper_flops_per_connection
    f = paper_flops_per_connection((203, 60, 26))
    assert round(f, 2) == 4.23
    assert abs(901 * f / 1000 - 3.8) < 0.05


# --------------------------------------------------------------------------- forward
@pytest.mark.parametrize("sizes", [(5, 3), (7, 1), (4, 6, 3), (5, 3, 4, 2)])
def test_forward_is_composition_of_logistic_models(sizes):
    x, _, w = _rand_case(sizes, 9, seed=11, scale=1.5)
    net = _net(sizes, w)
    y = net.forward(x)
    h = x.astype(np.float64)
    for Wl in net.layers(w):
        h = _logistic_layer(h, Wl)
    np.testing.assert_allclose(y, h, rtol=0, atol=1e-14)


def test_forward_zero_weights_gives_half():
    sizes = (6, 4, 3)
    net = _net(sizes, np.zeros(wl.num_weights(sizes)))
    y = net.forward(np.random.default_rng(0).uniform(-5, 5, (4, 6)).astype(np.float32))
    assert np.all(y == 0.5)


def test_forward_saturates_without_nan():
    sizes = (2, 1)
    w = np.array([1e4, -1e4, 0.0])
    y = _net(sizes, w).forward(np.array([[1, 0], [0, 1], [1, 1]], np.float32))
    assert y[0, 0] == 1.0 and y[1, 0] == 0.0 and y[2, 0] == 0.5


def test_onehot_forward_equals_dense_forward():
    w = wl.make_custom((203, 11, 5), 17, seed=3, onehot=True, init="uniform0.3")
    net = _net(w.sizes, w.weights)
    np.testing.assert_array_equal(net.forward(active=w.active), net.forward(x=w.dense_inputs()))


# --------------------------------------------------------------------------- gradient
def _half_sse(net, w, x, t):
    net.set_weights(w)
    y = net.forward(x)
    return 0.5 * np.sum((t.astype(np.float64) - y) ** 2)


# Nets of equal widths are included because there a mix-up of layers or a
# transposed weight block still has the right shape, so only the values can
# show it.
@pytest.mark.parametrize("sizes,n", [((3, 4, 2), 3), ((5, 3, 4, 2), 3), ((4, 1), 5), ((2, 7, 1), 4), ((3, 3, 3), 3),
                                     ((4, 4, 4, 4), 2)])
def test_summed_change_is_negative_gradient_central_differences(sizes, n):
    x, t, w = _rand_case(sizes, n, seed=sum(sizes) + n)
    net = _net(sizes, w)
    G, sse = net.gradient(t, x=x)
    probe = oracle.OracleNet(sizes, 64)
    h = 1e-5
    num = np.empty_like(G)
    for k in range(w.size):
        wp, wm = w.copy(), w.copy()
        wp[k] += h
        wm[k] -= h
        num[k] = (_half_sse(probe, wm, x, t) - _half_sse(probe, wp, x, t)) / (2 * h)
    scale = np.max(np.abs(num))
    assert scale > 1e-3
    assert np.max(np.abs(G - num)) <= 1e-7 * scale
    # The reported error is the summed squared difference (no factor 1/2).
    assert sse == pytest.approx(2 * _half_sse(probe, w, x, t), rel=1e-14)


def test_onehot_gradient_equals_dense_gradient():
    w = wl.make_custom((203, 9, 4), 13, seed=5, onehot=True, init="uniform0.3")
    net = _net(w.sizes, w.weights)
    g1, s1 = net.gradient(w.targets, active=w.active)
    g2, s2 = net.gradient(w.targets, x=w.dense_inputs())
    np.testing.assert_array_equal(g1, g2)
    assert s1 == s2


# --------------------------------------------------------------------------- update rule
def test_one_update_is_lr_times_summed_change():
    sizes, n = (4, 5, 3), 6
    x, t, w = _rand_case(sizes, n, seed=21)
    G, sse_g = _net(sizes, w).gradient(t, x=x)
    net = _net(sizes, w)
    sse = net.train_epoch(t, batch=n, lr=0.25, momentum=0.9, x=x)
    np.testing.assert_allclose(net.get_weights() - w, 0.25 * G, rtol=0, atol=1e-15)
    np.testing.assert_allclose(net.get_momentum(), 0.25 * G, rtol=0, atol=1e-15)
    # training-time error: measured with the weights of the batch's forward pass
    assert sse == sse_g


def test_momentum_carries_previous_change():
    # Two batches: V2 = lr * G2 + momentum * V1, W2 = W1 + V2 (classical momentum).
    sizes, n = (3, 4, 2), 8
    x, t, w = _rand_case(sizes, n, seed=31)
    lr, mom = 0.5, 0.75
    net = _net(sizes, w)
    net.train_epoch(t, batch=4, lr=lr, momentum=mom, x=x)
    G1, _ = _net(sizes, w).gradient(t[:4], x=x[:4])
    w1 = w + lr * G1
    G2, _ = _net(sizes, w1).gradient(t[4:], x=x[4:])
    v2 = lr * G2 + mom * (lr * G1)
    np.testing.assert_allclose(net.get_momentum(), v2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(net.get_weights(), w1 + v2, rtol=0, atol=1e-14)


def test_lr_zero_leaves_weights_unchanged():
    sizes = (5, 4, 3)
    x, t, w = _rand_case(sizes, 7, seed=41)
    for storage in (32, 64):
        net = _net(sizes, w, storage)
        w0 = net.get_weights()
        net.train_epoch(t, batch=3, lr=0.0, momentum=0.9, x=x)
        np.testing.assert_array_equal(net.get_weights(), w0)


def test_change_is_linear_in_lr_without_momentum():
    sizes = (4, 3, 2)
    x, t, w = _rand_case(sizes, 5, seed=51)
    d = []
    for lr in (0.125, 0.25):
        net = _net(sizes, w)
        net.train_epoch(t, batch=5, lr=lr, momentum=0.0, x=x)
        d.append(net.get_weights() - w)
    np.testing.assert_allclose(d[1], 2 * d[0], rtol=1e-12, atol=1e-16)


def test_closed_form_first_update_from_zero_weights():
    # All weights 0: every unit outputs 1/2, delta_L = (t - 1/2) / 4, hidden deltas
    # vanish (they are sums over zero weights), so only the last layer moves:
    # rows -> lr * sum_p (1/2)(t - 1/2)/4, bias row -> lr * sum_p (t - 1/2)/4.
    sizes, n, lr = (5, 4, 3), 6, 0.5
    g = np.random.default_rng(61)
    x = g.uniform(-1, 1, (n, 5)).astype(np.float32)
    t = np.where(g.random((n, 3)) < 0.5, 0.9, 0.1).astype(np.float32)
    net = _net(sizes, np.zeros(wl.num_weights(sizes)))
    sse = net.train_epoch(t, batch=n, lr=lr, momentum=0.9, x=x)
    t64 = t.astype(np.float64)
    assert sse == pytest.approx(np.sum((t64 - 0.5) ** 2), rel=1e-15)
    W0, W1 = net.layers(net.get_weights())
    assert np.all(W0 == 0)
    s = np.sum((t64 - 0.5) * 0.25, axis=0)
    np.testing.assert_allclose(W1[:4], np.tile(lr * 0.5 * s, (4, 1)), rtol=1e-15, atol=0)
    np.testing.assert_allclose(W1[4], lr * s, rtol=1e-15, atol=0)


def test_batch_sequencing_short_last_batch():
    # 5 patterns with batch 2 -> updates on [0,2), [2,4), [4,5) in order, momentum carried.
    sizes = (3, 3, 2)
    x, t, w = _rand_case(sizes, 5, seed=71)
    a = _net(sizes, w)
    sse_a, per = a.train_epoch(t, batch=2, lr=0.3, momentum=0.8, x=x, per_batch=True)
    b = _net(sizes, w)
    parts = [b.train_epoch(t[s:e], batch=2, lr=0.3, momentum=0.8, x=x[s:e]) for s, e in ((0, 2), (2, 4), (4, 5))]
    np.testing.assert_array_equal(a.get_weights(), b.get_weights())
    np.testing.assert_array_equal(a.get_momentum(), b.get_momentum())
    np.testing.assert_allclose(per, parts, rtol=1e-15)
    assert sse_a == pytest.approx(sum(parts), rel=1e-15)


def test_permutation_within_batch_only_changes_rounding():
    sizes = (6, 5, 3)
    x, t, w = _rand_case(sizes, 12, seed=81)
    perm = np.random.default_rng(1).permutation(12)
    a, b = _net(sizes, w), _net(sizes, w)
    a.train_epoch(t, batch=12, lr=0.2, momentum=0.9, x=x)
    b.train_epoch(t[perm], batch=12, lr=0.2, momentum=0.9, x=x[perm])
    np.testing.assert_allclose(a.get_weights(), b.get_weights(), rtol=0, atol=1e-14)


def test_identical_hidden_units_stay_identical():
    sizes = (4, 3, 2)
    x, t, w = _rand_case(sizes, 6, seed=91)
    net0 = oracle.OracleNet(sizes)
    W0, W1 = net0.layers(w.copy())
    W0[:, 2] = W0[:, 0]      # hidden unit 2 copies unit 0's incoming weights ...
    W1[2, :] = W1[0, :]      # ... and its outgoing weights
    w2 = np.concatenate([W0.ravel(), W1.ravel()])
    net = _net(sizes, w2)
    for _ in range(3):
        net.train_epoch(t, batch=3, lr=0.4, momentum=0.9, x=x)
    V0, V1 = net.layers(net.get_weights())
    np.testing.assert_array_equal(V0[:, 2], V0[:, 0])
    np.testing.assert_array_equal(V1[2, :], V1[0, :])


def test_single_pattern_small_step_lowers_its_error():
    sizes = (5, 4, 3)
    x, t, w = _rand_case(sizes, 1, seed=101)
    net = _net(sizes, w)
    e0 = net.train_epoch(t, batch=1, lr=1e-3, momentum=0.0, x=x)
    e1 = np.sum((t.astype(np.float64) - net.forward(x)) ** 2)
    assert e1 < e0


# --------------------------------------------------------------------------- precision / determinism
def test_float_storage_tracks_double_definition():
    w = wl.make("nettalk-80-b1024")
    d, f = _net(w.sizes, w.weights, 64), _net(w.sizes, w.weights, 32)
    sd = d.train_epoch(w.targets, w.batch, w.lr, w.momentum, active=w.active)
    sf = f.train_epoch(w.targets, w.batch, w.lr, w.momentum, active=w.active)
    assert abs(sf - sd) / sd < 1e-6
    wd, wf = d.get_weights(), f.get_weights()
    assert np.max(np.abs(wf - wd)) / np.max(np.abs(wd)) < 1e-6


def test_results_do_not_depend_on_thread_count():
    sizes = (9, 7, 4)
    x, t, w = _rand_case(sizes, 33, seed=111)
    res = []
    for nt in (1, 3):
        oracle.set_threads(nt)
        net = _net(sizes, w, 32)
        s = net.train_epoch(t, batch=8, lr=0.3, momentum=0.9, x=x)
        res.append((s, net.get_weights()))
    oracle.set_threads(0)
    assert res[0][0] == res[1][0]
    np.testing.assert_array_equal(res[0][1], res[1][1])


def test_rejects_bad_arguments():
    with pytest.raises(oracle.OracleError):
        oracle.OracleNet((5,))
    with pytest.raises(oracle.OracleError):
        oracle.OracleNet((5, 0, 2))
    net = oracle.OracleNet((10, 3, 2))
    t = np.zeros((2, 2), np.float32)
    with pytest.raises(oracle.OracleError):   # index out of range
        net.train_epoch(t, 2, 0.1, 0.9, active=np.array([[1, 10], [2, 3]]))
    with pytest.raises(oracle.OracleError):   # duplicate index within a pattern
        net.train_epoch(t, 2, 0.1, 0.9, active=np.array([[1, 1], [2, 3]]))
    with pytest.raises(oracle.OracleError):
        net.train_epoch(t, 0, 0.1, 0.9, x=np.zeros((2, 10), np.float32))


def test_every_pattern_presented_once_per_epoch():
    # With lr = 0 the epoch error is the summed squared error of the (pinned)
    # forward pass over ALL patterns, including a short last batch.
    sizes = (4, 3, 2)
    x, t, w = _rand_case(sizes, 7, seed=121)
    net = _net(sizes, w)
    sse = net.train_epoch(t, batch=3, lr=0.0, momentum=0.9, x=x)
    assert sse == pytest.approx(np.sum((t.astype(np.float64) - net.forward(x)) ** 2), rel=1e-14)


def test_short_batch_is_applied():
    sizes = (4, 3, 2)
    x, t, w = _rand_case(sizes, 1, seed=131)
    G, _ = _net(sizes, w).gradient(t, x=x)
    net = _net(sizes, w)
    net.train_epoch(t, batch=4, lr=0.5, momentum=0.9, x=x)
    np.testing.assert_allclose(net.get_weights(), w + 0.5 * G, rtol=0, atol=1e-15)
