"""The allocation-free training entry point (bp_train_batches_noalloc) against
bp_train_batches, through the C-ABI.

Both run the same launches over the same seeded inputs, one with the net's
own workspace and one with the per-GPU scratch array, so weights, momentum
and the epoch error must agree bit for bit.  Two calls in a row, the second
with a smaller input (fewer patterns, a smaller batch and a short last
batch): the scratch keeps the first call's contents, which the second must
not depend on.  Also: a call whose workspace exceeds the scratch is refused
and leaves the net unchanged.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_1801_01554_amd import bp
from paper_1801_01554_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "needs a ROCm device"
    bp.lib()
    return torch.device("cuda:0")


def _state(net):
    w = np.empty(net.n_weights, np.float32)
    v = np.empty(net.n_weights, np.float32)
    assert bp.bp_get_weights(net._h, w) == bp.BP_OK
    assert bp.bp_get_momentum(net._h, v) == bp.BP_OK
    return w, v


def _call(fn, net, x, t, n, batch, lr, mom):
    sse = ctypes.c_double(0.0)
    rc = fn(net._h, x.data_ptr(), t.data_ptr(), n, batch, lr, mom, sse)
    assert rc == bp.BP_OK, bp.bp_last_error(net._h)
    return sse.value


# (sizes, first call (patterns, batch), second call (patterns, batch)):
# split-K change products on the skinny kernel; three layers with ragged
# tiles; split-K change products on 128 x 128 tiles; the split-K output layer
CASES = [
    ((1030, 260, 70), (4200, 2100), (1500, 1100)),
    ((300, 129, 33, 5), (1000, 333), (200, 64)),
    ((2000, 2100, 6), (2200, 1100), (700, 300)),
    ((40, 3000, 300), (2000, 1000), (600, 500)),
]


@pytest.mark.parametrize("sizes,first,second", CASES)
def test_noalloc_matches_train_batches(dev, sizes, first, second):
    print(f"no-alloc vs bp_train_batches: sizes={sizes} first={first} second={second}", flush=True)
    n = max(first[0], second[0])
    w = wl.make_custom(sizes, n, seed=sum(sizes), onehot=False, input_kind="uniform", init="fanin")
    x = torch.from_numpy(w.inputs).to(dev)
    t = torch.from_numpy(w.targets).to(dev)
    ref, got = bp.Net(w.sizes), bp.Net(w.sizes)
    try:
        for net in (ref, got):
            net.set_weights(w.weights)
        for k, (np_, batch) in enumerate((first, second)):
            s_ref = _call(bp.bp_train_batches, ref, x, t, np_, batch, w.lr, w.momentum)
            s_got = _call(bp.bp_train_batches_noalloc, got, x, t, np_, batch, w.lr, w.momentum)
            torch.cuda.synchronize()
            wr, vr = _state(ref)
            wg, vg = _state(got)
            assert np.array_equal(wr.view(np.uint32), wg.view(np.uint32)), f"call {k}: weights differ"
            assert np.array_equal(vr.view(np.uint32), vg.view(np.uint32)), f"call {k}: momentum differs"
            assert s_ref == s_got, f"call {k}: error {s_ref} vs {s_got}"
    finally:
        ref.close()
        got.close()


def test_noalloc_refuses_workspace_beyond_scratch(dev):
    print("no-alloc: a batch whose workspace exceeds the scratch is refused", flush=True)
    sizes = (64, 4096, 4096, 8)
    n = 4096
    w = wl.make_custom(sizes, 8, seed=7, onehot=False, input_kind="uniform", init="fanin")
    net = bp.Net(w.sizes)
    try:
        net.set_weights(w.weights)
        x = torch.zeros((n, sizes[0]), dtype=torch.float32, device=dev)
        t = torch.zeros((n, sizes[-1]), dtype=torch.float32, device=dev)
        before = _state(net)
        rc = bp.bp_train_batches_noalloc(net._h, x.data_ptr(), t.data_ptr(), n, n, 0.1, 0.9, None)
        assert rc == bp.BP_EINVAL
        msg = bp.bp_last_error(net._h)
        assert "scratch" in msg and "bytes" in msg, msg
        after = _state(net)
        assert all(np.array_equal(a, b) for a, b in zip(before, after))
    finally:
        net.close()
