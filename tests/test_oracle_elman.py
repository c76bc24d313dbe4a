"""Pins of the oracle's Elman-net training (section 10.5).

The recurrent part is pinned to the already pinned feed-forward oracle by
doing its steps by hand in the test: the context inputs of each step are
assembled here from the hidden activations the feed-forward oracle reports
for the previous step, times the continuation flag; a window of steps is
then one pooled update of the feed-forward net over the unmasked patterns.
Further pins: no context reduces to plain pooled training over the patterns
in step order; a fully masked stream is the same as no stream; continuation
0 cuts the context; the training error equals the error of the forward
outputs when lr = 0.
"""
import numpy as np
import pytest

import oracle
from paper_1801_01554_amd import workloads as wl

SMALL = "elman-20+48-48-12"


def _seq(name=SMALL):
    return wl.make_sequences(name)


def _net(w, storage=32, context=True, sizes=None):
    n = oracle.OracleNet(sizes or w.sizes, storage)
    n.set_weights(w.weights.astype(np.float64))
    if context:
        n.set_context(w.ctx_layer, w.ctx_unit)
    return n


def test_no_context_is_pooled_training_in_step_order():
    w = _seq()
    s = w.spec
    sizes = (s.n_ext,) + s.hidden + (s.n_out,)
    g = np.random.default_rng(1)
    wt = g.uniform(-0.3, 0.3, wl.num_weights(sizes))
    a, b = oracle.OracleNet(sizes, 64), oracle.OracleNet(sizes, 64)
    a.set_weights(wt)
    b.set_weights(wt)
    ones = np.ones_like(w.mask)
    sa = a.train_sequences(w.inputs, w.targets, w.cont, ones, s.steps_per_update, 0.01, 0.9)
    T, S = w.cont.shape
    sb = b.train_epoch(w.targets.reshape(T * S, -1), s.steps_per_update * S, 0.01, 0.9,
                       x=w.inputs.reshape(T * S, -1))
    assert sa == sb
    np.testing.assert_array_equal(a.get_weights(), b.get_weights())


def test_context_matches_explicit_assembly_with_feedforward_oracle():
    w = _seq()
    s = w.spec
    T, S = w.cont.shape
    B, lr, mom = s.steps_per_update, 0.01, 0.9
    seq = _net(w, 32)
    sse_seq, win = seq.train_sequences(w.inputs, w.targets, w.cont, w.mask, B, lr, mom, per_window=True)

    ff = _net(w, 32, context=False)
    prev = np.zeros((S, s.n_ctx))
    win_ref = []
    for w0 in range(0, T, B):
        rows_x, rows_t = [], []
        for g in range(w0, min(T, w0 + B)):
            ctx = (w.cont[g][:, None].astype(np.float64) * prev).astype(np.float32)
            a0 = np.concatenate([w.inputs[g], ctx], axis=1)
            acts, _ = ff.batch_state(a0, w.targets[g])
            prev = acts[0][:, w.ctx_unit]                   # hidden layer 1 after this step
            keep = w.mask[g] != 0
            rows_x.append(a0[keep])
            rows_t.append(w.targets[g][keep])
        x, t = np.concatenate(rows_x), np.concatenate(rows_t)
        win_ref.append(ff.train_epoch(t, x.shape[0], lr, mom, x=x))
    np.testing.assert_array_equal(win, win_ref)
    np.testing.assert_array_equal(seq.get_weights(), ff.get_weights())
    np.testing.assert_array_equal(seq.get_momentum(), ff.get_momentum())


def test_masked_stream_is_no_stream():
    w = _seq()
    s = w.spec
    mask = w.mask.copy()
    mask[:, 0] = 0.0
    a, b = _net(w, 64), _net(w, 64)
    sa = a.train_sequences(w.inputs, w.targets, w.cont, mask, s.steps_per_update, 0.01, 0.9)
    sb = b.train_sequences(w.inputs[:, 1:], w.targets[:, 1:], w.cont[:, 1:], mask[:, 1:], s.steps_per_update,
                           0.01, 0.9)
    assert sa == sb
    np.testing.assert_array_equal(a.get_weights(), b.get_weights())


def test_continuation_zero_cuts_the_context():
    w = _seq()
    s = w.spec
    T, S = w.cont.shape
    net = _net(w, 64)
    y = net.forward_sequences(w.inputs, np.zeros_like(w.cont))
    ff = _net(w, 64, context=False)
    x0 = np.concatenate([w.inputs.reshape(T * S, -1), np.zeros((T * S, s.n_ctx), np.float32)], axis=1)
    np.testing.assert_array_equal(y.reshape(T * S, -1), ff.forward(x0))
    # with the real flags the context changes every continued step, and only those
    y1 = net.forward_sequences(w.inputs, w.cont)
    changed = np.any(y1 != y, axis=2)
    assert not changed[0].any()
    assert np.array_equal(changed, w.cont != 0)


def test_training_error_is_error_of_forward_outputs():
    w = _seq()
    s = w.spec
    net = _net(w, 64)
    y = net.forward_sequences(w.inputs, w.cont)
    ref = float(np.sum((w.mask[:, :, None].astype(np.float64) * (w.targets - y)) ** 2))
    sse = net.train_sequences(w.inputs, w.targets, w.cont, w.mask, s.steps_per_update, 0.0, 0.0)
    assert abs(sse - ref) <= 1e-12 * ref
    np.testing.assert_array_equal(net.get_weights(), w.weights.astype(np.float64))


def test_context_arguments_are_checked():
    net = oracle.OracleNet((10, 4, 2), 64)
    for fl, fu in (([0], [0]), ([2], [0]), ([1], [4]), ([1] * 11, [0] * 11)):
        with pytest.raises(oracle.OracleError):
            net.set_context(fl, fu)
    with pytest.raises(oracle.OracleError):
        oracle.OracleNet((10, 2), 64).set_context([1], [0])      # no hidden layer
    net.set_context([1, 1], [3, 0])
    net.set_context([], [])
