"""Pins of the oracle's optional parts: the table sigmoid (section 4.3), the
range check of the summed changes (section 8) and the checkpoint guard
(section 10.4).

As for the core method, no test retypes the oracle's formulas:

* the table sigmoid is pinned to the interpolation error bound of a piecewise
  linear interpolant (h^2 / 8 max |sigma''|, with max |sigma''| = 1 / (6 sqrt 3)
  for the logistic), to exact values at the table's nodes, to its end values,
  symmetry, monotonicity and linearity between nodes;
* the range check is pinned to closed-form fault counts when one pattern's
  target is poisoned (which summed changes that pattern reaches follows from
  the structure of the method), to "no effect" with a generous limit and to
  "momentum only" with a limit below every change;
* the guard is pinned to a hand-worked decision sequence and to the paper's
  claim that a rollback makes training immune to a transient corruption.
"""
import numpy as np
import pytest

import oracle
from paper_1801_01554_amd import workloads as wl

H_TABLE = 30.0 / 255.0                                   # node spacing of the table
SIGMA2_MAX = 1.0 / (6.0 * np.sqrt(3.0))                  # max |sigma''| of the logistic
INTERP_BOUND = H_TABLE ** 2 / 8.0 * SIGMA2_MAX           # 1.6648e-4
# The index and fraction are formed in single precision: (z + 15) is rounded
# to a float below 32 (ulp 2^-19) and x1 = 8.5 (z + 15) to a float below 256
# (ulp 2^-16), moving the interpolation point by at most (2^-20 + 2^-17 / 8.5)
# in z, times the largest slope 1/4.
POSITION_ROUNDING = 0.25 * (2.0 ** -20 + 2.0 ** -17 / 8.5)


def _sig(z):
    return 1.0 / (1.0 + np.exp(-np.asarray(z, np.float64)))


def _table_net(storage=64):
    n = oracle.OracleNet((3, 2, 1), storage)
    n.set_sigmoid(oracle.OracleNet.SIGMOID_TABLE)
    return n


# --------------------------------------------------------------------------- table sigmoid
def test_table_sigmoid_error_meets_interpolation_bound():
    z = np.linspace(-20.0, 20.0, 800001)
    err = np.abs(_table_net().eval_sigmoid(z) - _sig(z))
    assert err.max() <= INTERP_BOUND + POSITION_ROUNDING + 1e-12
    # the bound is attained near the inflection points of sigma'' (|z| ~ 1.317)
    assert err.max() >= 0.99 * INTERP_BOUND
    assert 1.0 < abs(z[np.argmax(err)]) < 1.6


def test_table_sigmoid_is_exact_at_nodes():
    # z = -15 + 2k maps to x1 = 17k exactly, a table node
    z = -15.0 + 2.0 * np.arange(16)
    np.testing.assert_array_equal(_table_net().eval_sigmoid(z), _sig(z))
    # float storage: the node value rounded to float
    np.testing.assert_array_equal(_table_net(32).eval_sigmoid(z), _sig(z).astype(np.float32).astype(np.float64))


def test_table_sigmoid_ends_and_nan():
    net = _table_net()
    lo, hi = _sig(-15.0), _sig(15.0)
    y = net.eval_sigmoid([-15.0, -15.5, -1e6, -np.inf, 15.0, 15.01, 1e30, np.inf])
    np.testing.assert_array_equal(y, [lo, lo, lo, lo, hi, hi, hi, hi])
    assert np.isnan(net.eval_sigmoid([np.nan])[0])


def test_table_sigmoid_symmetric_and_monotone():
    z = np.linspace(0.0, 16.0, 200001)
    net = _table_net()
    yp, ym = net.eval_sigmoid(z), net.eval_sigmoid(-z)
    assert np.abs(yp + ym - 1.0).max() < 1e-6
    y = net.eval_sigmoid(np.linspace(-16, 16, 400001))
    assert np.all(np.diff(y) >= 0.0)


def test_table_sigmoid_is_linear_between_nodes():
    # node i at x1 = i; points strictly inside one interval lie on one line
    net = _table_net()
    for i in (3, 100, 137, 200, 254):
        zlo = i / 8.5 - 15.0
        z = zlo + np.linspace(0.05, 0.95, 19) / 8.5
        y = net.eval_sigmoid(z)
        slope = np.diff(y) / np.diff(z)
        # each point's position is rounded by at most dz (single precision), so
        # adjacent-point slopes agree to 2 dz / spacing, relative
        dz = 2.0 ** -20 + 2.0 ** -17 / 8.5
        assert np.ptp(slope) <= 2 * (2 * dz / np.diff(z).min()) * abs(slope).max() + 1e-9
        # and the line joins the two node values
        a, b = _sig(zlo), _sig(zlo + 1 / 8.5)
        assert abs(y[9] - (a + (b - a) * (z[9] - zlo) * 8.5)) < 3e-7


def test_table_sigmoid_net_tracks_exact_net():
    # the whole forward pass with the table stays within the per-unit bound
    sizes = (6, 5, 4)
    g = np.random.default_rng(3)
    x = g.uniform(-1, 1, (20, 6)).astype(np.float32)
    w = g.uniform(-1, 1, wl.num_weights(sizes))
    a, b = oracle.OracleNet(sizes), oracle.OracleNet(sizes)
    a.set_weights(w)
    b.set_weights(w)
    b.set_sigmoid(1)
    d = np.abs(a.forward(x) - b.forward(x)).max()
    # hidden error <= bound, propagated through <= 5 weights of |w| <= 1 and slope <= 1/4
    assert 0 < d <= (1 + 5 * 0.25) * (INTERP_BOUND + POSITION_ROUNDING)


# --------------------------------------------------------------------------- range check
def _dense_case(sizes, n, seed):
    g = np.random.default_rng(seed)
    x = g.uniform(-1, 1, (n, sizes[0])).astype(np.float32)
    t = np.where(g.random((n, sizes[-1])) < 0.5, 0.9, 0.1).astype(np.float32)
    w = g.uniform(-0.5, 0.5, wl.num_weights(sizes)).astype(np.float32).astype(np.float64)
    return x, t, w


def _trained(sizes, w, x, t, limit, lr=0.5, mom=0.9, batch=None, storage=32, active=None):
    net = oracle.OracleNet(sizes, storage)
    net.set_weights(w)
    if limit is not None:
        net.set_fault_limit(limit)
    n = t.shape[0]
    if active is not None:
        net.train_epoch(t, batch or n, lr, mom, active=active)
    else:
        net.train_epoch(t, batch or n, lr, mom, x=x)
    return net


def test_generous_limit_changes_nothing():
    sizes = (6, 5, 3)
    x, t, w = _dense_case(sizes, 12, 1)
    a = _trained(sizes, w, x, t, None, batch=4)
    b = _trained(sizes, w, x, t, 1e30, batch=4)
    np.testing.assert_array_equal(a.get_weights(), b.get_weights())
    np.testing.assert_array_equal(a.get_momentum(), b.get_momentum())
    assert b.fault_count() == 0


@pytest.mark.parametrize("poison", [np.nan, 1e30])
def test_poisoned_target_faults_exactly_what_it_reaches_dense(poison):
    # A poisoned target k of pattern p makes delta_2[p][k] huge (or NaN), which
    # reaches G1[:, k] (H + 1 entries) and, through delta_1[p][:] (every hidden
    # unit, since W1[:, k] != 0), every entry of G0 whose input a_0[p][i] != 0
    # plus the bias row: (n0 + 1) * H.  Nothing else.
    sizes = (6, 5, 3)
    n0, H, O = sizes
    x, t, w = _dense_case(sizes, 8, 2)
    p, k = 3, 1
    tp = t.copy()
    tp[p, k] = poison
    net = _trained(sizes, w, x, tp, 1e6, lr=0.5, mom=0.9)
    assert net.fault_count() == (H + 1) + (n0 + 1) * H
    W0, W1 = net.layers(net.get_weights())
    W0i, W1i = net.layers(w.astype(np.float32).astype(np.float64))
    # faulted entries: V = 0 * lr + mom * 0 -> weight unchanged
    np.testing.assert_array_equal(W0, W0i)
    np.testing.assert_array_equal(W1[:, k], W1i[:, k])
    # the other output columns see only finite deltas: same as with a clean target
    tc = t.copy()
    tc[p, k] = 0.5
    clean = _trained(sizes, w, x, tc, None, lr=0.5, mom=0.9)
    C1 = clean.layers(clean.get_weights())[1]
    other = [c for c in range(O) if c != k]
    np.testing.assert_array_equal(W1[:, other], C1[:, other])


@pytest.mark.parametrize("poison", [np.nan, 1e30])
def test_poisoned_target_faults_only_active_rows_onehot(poison):
    # One-hot inputs: delta_1[p] reaches only the n_active rows of pattern p
    # and the bias row of W0: (n_active + 1) * H faults there, plus G1[:, k].
    # (Inactive inputs take no part, so a NaN delta does not reach their rows.)
    n0, H, O, k_act = 30, 6, 4, 3
    sizes = (n0, H, O)
    g = np.random.default_rng(5)
    act = np.stack([g.choice(n0, k_act, replace=False) for _ in range(10)]).astype(np.int32)
    t = np.where(g.random((10, O)) < 0.5, 0.9, 0.1).astype(np.float32)
    w = g.uniform(-0.5, 0.5, wl.num_weights(sizes))
    t[7, 2] = poison
    net = _trained(sizes, w, None, t, 1e6, active=act)
    assert net.fault_count() == (H + 1) + (k_act + 1) * H


def test_tiny_limit_faults_every_nonzero_change_onehot():
    # Rows of W0 no pattern of the batch activates have G = 0 exactly (in range);
    # every other summed change is nonzero and faults.
    n0, H, O, k_act = 40, 5, 3, 2
    sizes = (n0, H, O)
    g = np.random.default_rng(6)
    act = np.stack([g.choice(20, k_act, replace=False) for _ in range(9)]).astype(np.int32)  # rows >= 20 unused
    t = np.where(g.random((9, O)) < 0.5, 0.9, 0.1).astype(np.float32)
    w = g.uniform(-0.5, 0.5, wl.num_weights(sizes))
    unused = n0 - len(np.unique(act))
    net = _trained(sizes, w, None, t, 1e-30, active=act)
    assert net.fault_count() == wl.num_weights(sizes) - unused * H


def test_all_faulted_batch_moves_by_momentum_only():
    sizes = (5, 4, 2)
    x, t, w = _dense_case(sizes, 6, 7)
    net = oracle.OracleNet(sizes, 32)
    net.set_weights(w)
    net.train_epoch(t[:3], 3, 0.5, 0.9, x=x[:3])          # clean first update: V != 0
    W1, V1 = net.get_weights(), net.get_momentum()
    assert np.count_nonzero(V1) == V1.size
    net.set_fault_limit(1e-30)
    net.train_epoch(t[3:], 3, 0.5, 0.9, x=x[3:])
    assert net.fault_count() == wl.num_weights(sizes)
    # V = 0 * lr + mom * V, then W += V, each rounded to float storage
    v2 = (0.9 * V1).astype(np.float32).astype(np.float64)
    np.testing.assert_array_equal(net.get_momentum(), v2)
    np.testing.assert_array_equal(net.get_weights(), (W1 + v2).astype(np.float32).astype(np.float64))


def test_fault_limit_rejects_bad_values():
    net = oracle.OracleNet((2, 2), 32)
    for bad in (-1.0, np.nan):
        with pytest.raises(oracle.OracleError):
            net.set_fault_limit(bad)


# --------------------------------------------------------------------------- checkpoint guard
def test_guard_decisions_hand_worked():
    sizes = (2, 1)
    net = oracle.OracleNet(sizes, 64)
    A, B, C = np.full(3, 1.0), np.full(3, 2.0), np.full(3, 3.0)
    net.set_weights(A)
    net.guard_config(every=2, jump=1.5)                 # checkpoint = A
    assert net.guard_epoch(10.0) == 0                   # accepted (nothing to compare)
    net.set_weights(B)
    assert net.guard_epoch(8.0) == 0                    # accepted; 2nd -> checkpoint = B (error 8)
    net.set_weights(C)
    assert net.guard_epoch(20.0) == 1                   # 20 > 1.5 * 8: back to B
    np.testing.assert_array_equal(net.get_weights(), B)
    assert net.guard_epoch(20.0) == 0                   # same jump at the same epoch: accepted
    net.set_weights(C)
    assert net.guard_epoch(29.0) == 0                   # 29 <= 1.5 * 20; 2nd -> checkpoint = C (error 29)
    net.set_weights(A)
    assert net.guard_epoch(float("nan")) == 1           # not a number counts as a jump: back to C
    np.testing.assert_array_equal(net.get_weights(), C)
    assert net.guard_epoch(43.0) == 0                   # 43 <= 1.5 * 29


def test_rollback_makes_training_immune_to_transient_corruption():
    # Section 10.4: restoring a checkpoint after an error jump and training on
    # gives the same net as a run that was never corrupted (training is
    # deterministic, so the replayed epochs are identical).
    sizes = (6, 5, 3)
    x, t, w = _dense_case(sizes, 24, 8)
    args = dict(batch=6, lr=0.3, momentum=0.9, x=x)

    clean = oracle.OracleNet(sizes, 32)
    clean.set_weights(w)
    sse_clean = [clean.train_epoch(t, **args) for _ in range(6)]

    net = oracle.OracleNet(sizes, 32)
    net.set_weights(w)
    net.guard_config(every=2, jump=1.5)
    accepted, rollbacks = [], 0
    while len(accepted) < 6:
        if len(accepted) == 3 and rollbacks == 0:
            bad = net.get_weights()
            bad[::3] = 40.0                              # a transient corruption of the weights
            v = net.get_momentum()
            net.set_weights(bad)
            net.set_momentum(v)
        sse = net.train_epoch(t, **args)
        if net.guard_epoch(sse):
            rollbacks += 1
            accepted = accepted[: len(accepted) - (len(accepted) % 2)]   # back to the last checkpoint
            continue
        accepted.append(sse)
    assert rollbacks == 1
    assert accepted == sse_clean
    np.testing.assert_array_equal(net.get_weights(), clean.get_weights())
    np.testing.assert_array_equal(net.get_momentum(), clean.get_momentum())


def test_guard_rejects_bad_arguments():
    net = oracle.OracleNet((2, 1), 32)
    with pytest.raises(oracle.OracleError):
        net.guard_epoch(1.0)
    with pytest.raises(oracle.OracleError):
        net.guard_config(0, 1.5)
    with pytest.raises(oracle.OracleError):
        net.guard_config(1, 0.0)


def test_onehot_first_layer_uses_only_active_rows():
    # A non-finite weight in a row no pattern activates leaves one-hot outputs
    # finite (the gather takes only the active rows), while the same inputs
    # given densely meet it as 0 * NaN.
    n0, H, O = 12, 4, 3
    sizes = (n0, H, O)
    g = np.random.default_rng(9)
    act = np.array([[0, 3, 5], [1, 3, 7], [2, 4, 6]], np.int32)
    w = g.uniform(-0.5, 0.5, wl.num_weights(sizes))
    w[11 * H + 2] = np.nan                              # W0[11][2], row 11 never active
    net = oracle.OracleNet(sizes, 64)
    net.set_weights(w)
    assert np.all(np.isfinite(net.forward(active=act)))
    assert np.all(np.isnan(net.forward(x=wl.dense_from_active(act, n0))))
