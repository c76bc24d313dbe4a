"""Writes the stored expected values under tests/golden/ (calls only the oracle).

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
    if what == "epoch":
        for nm in sys.argv[2:]:
            epoch(nm)
    else:
        raise SystemExit(__doc__)
