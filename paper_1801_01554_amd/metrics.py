"""Work counts used to report throughput (host-side bookkeeping only).

* Connections W: every weight including the bias ("true unit") rows
  (section 6.3 counts 13,826 for the 203-60-26 NETtalk net).
* Connections per second: W x patterns presented / wall time (section 7.1);
  it counts neither how often weights are updated nor that input connections
  need less work.
* The paper's MCPS-to-MFLOPS factor 4 + 2 (W - W_i) / W (section 7.2), with
  W_i the weights leaving the input layer.
"""
from __future__ import annotations

from typing import Sequence


def num_weights(sizes: Sequence[int]) -> int:
    return int(sum((sizes[l] + 1) * sizes[l + 1] for l in range(len(sizes) - 1)))


def input_weights(sizes: Sequence[int]) -> int:
    return int((sizes[0] + 1) * sizes[1])


def paper_flops_per_connection(sizes: Sequence[int]) -> float:
    """Flops per connection per pattern by the paper's conversion (forward + backward, no update)."""
    w, wi = num_weights(sizes), input_weights(sizes)
    return 4.0 + 2.0 * (w - wi) / w


def dense_flops_per_pattern(sizes: Sequence[int], batch: int) -> float:
    """Algorithmic flops per pattern of the dense path.

    2W (forward) + 2W (batch sum of the changes, bias rows included)
    + 2 * sum_{l>=1} n_l n_{l+1} (hidden deltas) + 4W / batch (lr and momentum update).
    """
    w = num_weights(sizes)
    bwd = sum(2 * sizes[l] * sizes[l + 1] for l in range(1, len(sizes) - 1))
    return 2.0 * w + 2.0 * w + bwd + 4.0 * w / batch


def gemm_flops_per_batch(sizes: Sequence[int], rows: int) -> float:
    """Matrix-product flops of one pooled update over `rows` patterns (dense path).

    forward l: 2 rows n_l n_{l+1}; hidden deltas l >= 1: 2 rows n_{l+1} n_l;
    change sums: 2 rows n_l n_{l+1} (the bias row is a column sum, not counted here).
    """
    f = 0.0
    for l in range(len(sizes) - 1):
        mn = sizes[l] * sizes[l + 1]
        f += 2.0 * rows * mn * (3 if l >= 1 else 2)
    return f


def onehot_bytes_per_update(sizes: Sequence[int]) -> float:
    """Algorithmic HBM bytes of the weight state per update: read W, V; write W, V (fp32)."""
    return 16.0 * num_weights(sizes)


def onehot_bytes_per_pattern(sizes: Sequence[int], n_active: int) -> float:
    """Algorithmic HBM bytes of the data per pattern: int32 active indices + fp32 targets."""
    return 4.0 * n_active + 4.0 * sizes[-1]
