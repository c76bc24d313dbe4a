"""Writes the stored expected values under tests/golden/ (calls only the oracle).

    python tests/golden/make_golden.py worked            # 2-2-1 worked example
    python tests/golden/make_golden.py epoch NAME [...]   # full-epoch errors of a named workload

Every number written here comes from ``oracle/`` on inputs from the seeded
generators; nothing comes from the HIP library.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_1801_01554_amd import workloads as wl  # noqa: E402

# A 2-2-1 net, two patterns in one batch, two consecutive updates.
WORKED = {
    "sizes": [2, 2, 1],
    "weights": [0.1, -0.2, 0.3, 0.4, 0.0, 0.1, 0.5, -0.6, 0.2],
    "inputs": [[1.0, 0.0], [0.0, 1.0]],
    "targets": [[0.9], [0.1]],
    "lr": 0.5,
    "momentum": 0.9,
    "batch": 2,
}


def worked():
    c = WORKED
    net = oracle.OracleNet(c["sizes"], 64)
    net.set_weights(np.array(c["weights"], np.float64))
    x = np.array(c["inputs"], np.float32)
    t = np.array(c["targets"], np.float32)
    steps = []
    for _ in range(2):
        y = net.forward(x)[:, 0].tolist()
        sse = net.train_epoch(t, c["batch"], c["lr"], c["momentum"], x=x)
        steps.append({"outputs_before": y, "sse": sse, "weights_after": net.get_weights().tolist(),
                      "momentum_after": net.get_momentum().tolist()})
    out = dict(c, steps=steps,
               source="oracle/ (double storage) via tests/golden/make_golden.py worked")
    # The float inputs 0.9 / 0.1 are rounded to float32 before use.
    with open(os.path.join(HERE, "worked_2_2_1.json"), "w") as f:
        json.dump(out, f, indent=1)
    print("wrote worked_2_2_1.json")


def epoch(name, storages=(64, 32)):
    w = wl.make(name)
    s = w.spec
    res = {"workload": name, "sizes": list(s.sizes), "n_patterns": s.n_patterns, "batch": s.batch,
           "lr": w.lr, "momentum": w.momentum, "epochs": s.epochs,
           "source": "oracle/ via tests/golden/make_golden.py epoch", "threads": oracle.get_threads()}
    for bits in storages:
        net = oracle.OracleNet(w.sizes, bits)
        net.set_weights(w.weights)
        ep, per = [], []
        t0 = time.time()
        for e in range(s.epochs):
            kw = {"active": w.active} if w.active is not None else {"x": w.inputs}
            sse, pb = net.train_epoch(w.targets, s.batch, w.lr, w.momentum, per_batch=True, **kw)
            ep.append(sse)
            per.append(pb.tolist())
            print(f"{name} storage{bits} epoch {e} sse {sse:.10g} ({time.time() - t0:.0f}s)", flush=True)
        wts = net.get_weights()
        g = np.random.default_rng(12345)
        idx = np.sort(g.choice(wts.size, size=min(4096, wts.size), replace=False))
        res[f"storage{bits}"] = {
            "epoch_sse": ep, "batch_sse": per, "seconds": time.time() - t0,
            "final_weight_sample_index": idx.tolist(), "final_weight_sample": wts[idx].tolist(),
            "final_weight_absmax": float(np.max(np.abs(wts))),
        }
    with open(os.path.join(HERE, f"epoch_{name}.json"), "w") as f:
        json.dump(res, f)
    print(f"wrote epoch_{name}.json")


if __name__ == "__main__":
    what = sys.argv[1]
    if what == "worked":
        worked()
    elif what == "epoch":
        for nm in sys.argv[2:]:
            epoch(nm)
    else:
        raise SystemExit(__doc__)
