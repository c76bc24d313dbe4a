"""Graph replay of repeated training calls against direct launches.

The second of two training calls with the same arguments is captured into a
HIP graph and later such calls replay it.  Replays run the same kernels with
the same arguments, so every call must give bit-identical weights, momenta,
error and forward outputs to a net that launches every kernel directly.
Each case interleaves the replays with the program's own eager work (a
forward pass, host copies, synchronisations), changes an argument (the
learning rate: a new capture) and an option (the table sigmoid: the
captured graph is dropped), and covers the fused small-net path, the dense
generic path and the one-hot generic path.  Calls of a single batch always
launch directly; their case checks that the replay setting leaves them so.
"""
import numpy as np
import pytest
import torch

from paper_1801_01554_amd import bp
from paper_1801_01554_amd import workloads as wl
from parity_util import to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU graph tests need a ROCm device"
    bp.lib()
    return torch.device("cuda:0")


def _say(msg):
    print(msg, flush=True)


# (lr, table sigmoid) per call: calls 1-4 capture at call 2 and replay, call
# 5 has a new lr (direct), 6 captures it, 7 replays, 8 switches to the table
# sigmoid (graph dropped, direct), 9 captures, 10 replays.
CALLS = [(0.05, False)] * 4 + [(0.02, False)] * 3 + [(0.02, True)] * 3

CASES = [
    ("fused small-net path", (203, 120, 26), 2048, 512, True),
    ("dense generic path", (64, 96, 10), 3000, 1024, False),
    ("one-hot generic path", (60, 40, 30, 12), 1500, 256, True),
    ("single batch per call (direct launches)", (203, 120, 26), 512, 512, True),
]


def _run(w, batch, dev, replay):
    net = bp.Net(w.sizes)
    net.set_weights(w.weights)
    net.set_graph_replay(replay)
    x, a, t = to_device(w, dev)
    kw = {"active": a} if a is not None else {"inputs": x}
    outs = []
    table_on = False
    for lr, table in CALLS:
        if table != table_on:
            net.set_sigmoid(bp.BP_SIGMOID_TABLE if table else bp.BP_SIGMOID_EXACT)
            table_on = table
        sse = net.train_batches(t, batch, lr, 0.9, **kw)
        y = net.forward(**kw).cpu().numpy()          # eager work between replays
        torch.cuda.synchronize()
        outs.append((sse, net.get_weights(), net.get_momentum(), y))
    net.close()
    return outs


@pytest.mark.parametrize("name,sizes,n,batch,onehot", CASES)
def test_replay_matches_direct_launches(dev, name, sizes, n, batch, onehot):
    _say(f"case graph replay {name}: sizes={sizes} n={n} batch={batch}")
    w = wl.make_custom(sizes, n, seed=97, onehot=onehot)
    direct = _run(w, batch, dev, False)
    replay = _run(w, batch, dev, True)
    for k, (d, r) in enumerate(zip(direct, replay)):
        _say(f"  call {k}: sse direct {d[0]} replay {r[0]}")
        assert d[0] == r[0]
        np.testing.assert_array_equal(d[1], r[1])
        np.testing.assert_array_equal(d[2], r[2])
        np.testing.assert_array_equal(d[3], r[3])


def test_replay_reads_buffers_at_replay_time(dev):
    """A replayed call sees new contents of the same argument buffers."""
    w = wl.make_custom((203, 120, 26), 1024, seed=98, onehot=True)
    _, a, t = to_device(w, dev)
    nets = [bp.Net(w.sizes) for _ in range(2)]
    for net, on in zip(nets, (False, True)):
        net.set_weights(w.weights)
        net.set_graph_replay(on)
    for k in range(4):
        t.copy_(torch.from_numpy(np.roll(w.targets, k, axis=0)).to(dev))   # same buffer, new targets
        s = [net.train_batches(t, 256, 0.05, 0.9, active=a) for net in nets]
        _say(f"  call {k}: sse direct {s[0]} replay {s[1]}")
        assert s[0] == s[1]
        np.testing.assert_array_equal(nets[0].get_weights(), nets[1].get_weights())
    for net in nets:
        net.close()
