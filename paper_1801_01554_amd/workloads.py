"""Seeded synthetic inputs for pooled back-propagation.

This module only draws numbers: it holds none of the method's arithmetic.
The same arrays feed the CPU oracle (tests only) and the HIP path, so that
both sides see bit-identical inputs.

The named workloads stand in for the paper's NETtalk benchmark (section
6.3: a 203-input window of 7 letter positions x 29 symbols, one-hot coded,
26 output bits), which is not available here, and add two larger dense nets
that make the weight contractions GEMM-bound.  Recipe (all generated in
float64 and rounded to float32 once):

* three independent PCG64 streams per workload seed: inputs, targets,
  weights (``default_rng([seed, k])`` for k = 0, 1, 2);
* one-hot inputs: ``sym = integers(0, 29, (N, 7))``, active index
  ``29 * position + sym`` (exactly 7 ones among 203 inputs);
* dense inputs: ``uniform(-1, 1)`` or ``standard_normal()``, row-major;
* targets: ``random() < p`` mapped to 0.9 / 0.1 (p = 0.15 one-hot, 0.5 dense);
* weights, layer by layer in the flat C-ABI layout (rows input-major, the
  bias row last): ``uniform(-r, r)`` with r = 0.3 (one-hot nets) or
  1/sqrt(fan_in) (dense nets, fan_in excluding the bias).

Large arrays are drawn in row chunks from the same stream, which yields the
same values as one draw; ``n_patterns`` takes a prefix of the full set.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

N_POS = 7      # letter positions in the input window
N_SYM = 29     # symbols per position
CHUNK_ROWS = 16384


@dataclasses.dataclass(frozen=True)
class Spec:
    name: str
    sizes: tuple            # layer sizes n_0 .. n_L
    onehot: bool            # inputs given as active indices
    n_patterns: int
    batch: int
    lr: float
    momentum: float
    epochs: int
    seed: int
    input_kind: str         # "onehot", "uniform", "normal"
    target_p: float         # probability of a 0.9 target bit
    init: str               # "uniform0.3" or "fanin"
    note: str = ""


SPECS = {
    s.name: s
    for s in [
        Spec("nettalk-80-b1024", (203, 80, 26), True, 1024, 1024, 0.1, 0.9, 1, 1,
             "onehot", 0.15, "uniform0.3", "tiny NETtalk-shaped net, one update"),
        Spec("nettalk-120-b512", (203, 120, 26), True, 20000, 512, 0.05, 0.9, 10, 2,
             "onehot", 0.15, "uniform0.3", "NETtalk-shaped net, 40 updates per epoch"),
        Spec("nettalk-120-b16", (203, 120, 26), True, 20000, 16, 0.02, 0.9, 2, 2,
             "onehot", 0.15, "uniform0.3", "small-batch latency case, 1250 updates per epoch"),
        Spec("wide-1024-4096-1024", (1024, 4096, 1024), False, 262144, 4096, 0.01, 0.9, 1, 4,
             "uniform", 0.5, "fanin", "wide dense net, GEMM-bound"),
        Spec("deep-512-2048x3-64", (512, 2048, 2048, 2048, 64), False, 524288, 8192, 0.01, 0.9, 1, 5,
             "normal", 0.5, "fanin", "deep dense net, multi-layer delta chaining"),
    ]
}
# The order the workloads are listed in (smallest first).
ORDER = list(SPECS)


@dataclasses.dataclass
class Workload:
    spec: Spec
    sizes: tuple
    n_patterns: int
    inputs: Optional[np.ndarray]    # float32 [n][n0] (dense) or None
    active: Optional[np.ndarray]    # int32 [n][7] (one-hot) or None
    targets: np.ndarray             # float32 [n][nL]
    weights: np.ndarray             # float32 flat, C-ABI layout

    @property
    def batch(self) -> int:
        return self.spec.batch

    @property
    def lr(self) -> float:
        return float(np.float32(self.spec.lr))

    @property
    def momentum(self) -> float:
        return float(np.float32(self.spec.momentum))

    def dense_inputs(self) -> np.ndarray:
        """Inputs as a float32 [n][n0] matrix (0/1 for one-hot workloads)."""
        if self.inputs is not None:
            return self.inputs
        return dense_from_active(self.active, self.sizes[0])


def num_weights(sizes: Sequence[int]) -> int:
    """Connection count including the bias ("true unit") rows."""
    return int(sum((sizes[i] + 1) * sizes[i + 1] for i in range(len(sizes) - 1)))


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def _draw_rows(draw, n_rows: int, n_cols: int, dtype=np.float32) -> np.ndarray:
    out = np.empty((n_rows, n_cols), dtype=dtype)
    for r0 in range(0, n_rows, CHUNK_ROWS):
        r1 = min(n_rows, r0 + CHUNK_ROWS)
        out[r0:r1] = draw((r1 - r0, n_cols))
    return out


def draw_inputs(kind: str, seed: int, n: int, n0: int):
    """Returns (dense float32 [n][n0] or None, active int32 [n][7] or None)."""
    g = _rng(seed, 0)
    if kind == "onehot":
        if n0 != N_POS * N_SYM:
            raise ValueError("one-hot window inputs need n0 = 7 * 29")
        sym = g.integers(0, N_SYM, size=(n, N_POS), dtype=np.int64)
        act = (sym + N_SYM * np.arange(N_POS, dtype=np.int64)[None, :]).astype(np.int32)
        return None, act
    if kind == "uniform":
        return _draw_rows(lambda s: g.uniform(-1.0, 1.0, size=s), n, n0), None
    if kind == "normal":
        return _draw_rows(lambda s: g.standard_normal(size=s), n, n0), None
    raise ValueError(kind)


def draw_targets(seed: int, n: int, n_out: int, p: float) -> np.ndarray:
    g = _rng(seed, 1)
    return _draw_rows(lambda s: np.where(g.random(size=s) < p, 0.9, 0.1), n, n_out)


def draw_weights(seed: int, sizes: Sequence[int], init: str) -> np.ndarray:
    g = _rng(seed, 2)
    parts = []
    for l in range(len(sizes) - 1):
        rows, cols = sizes[l] + 1, sizes[l + 1]
        r = 0.3 if init == "uniform0.3" else 1.0 / np.sqrt(sizes[l])
        parts.append(g.uniform(-r, r, size=rows * cols).astype(np.float32))
    return np.concatenate(parts)


def make(name: str, n_patterns: Optional[int] = None) -> Workload:
    """Builds a named workload; ``n_patterns`` keeps only the first patterns."""
    s = SPECS[name]
    n = s.n_patterns if n_patterns is None else int(n_patterns)
    if n < 0 or n > s.n_patterns:
        raise ValueError(f"n_patterns must be in [0, {s.n_patterns}]")
    x, act = draw_inputs(s.input_kind, s.seed, n, s.sizes[0])
    t = draw_targets(s.seed, n, s.sizes[-1], s.target_p)
    w = draw_weights(s.seed, s.sizes, s.init)
    return Workload(s, tuple(s.sizes), n, x, act, t, w)


def make_custom(sizes: Sequence[int], n: int, seed: int, onehot: bool = False,
                input_kind: str = "uniform", target_p: float = 0.5,
                init: str = "fanin") -> Workload:
    """A small ad-hoc workload with the same recipe (tests use it for ragged shapes).

    For ``onehot=True`` the input layer may have any size n0 >= 7: the active
    indices are 7 distinct values drawn uniformly from [0, n0).
    """
    sizes = tuple(int(v) for v in sizes)
    g = _rng(seed, 0)
    if onehot:
        n0 = sizes[0]
        if n0 == N_POS * N_SYM:
            x, act = draw_inputs("onehot", seed, n, n0)
        else:
            k = min(N_POS, n0)
            act = np.stack([g.permutation(n0)[:k] for _ in range(n)]).astype(np.int32) \
                if n > 0 else np.zeros((0, k), np.int32)
            x = None
    else:
        x, act = draw_inputs(input_kind, seed, n, sizes[0])
    t = draw_targets(seed, n, sizes[-1], target_p)
    w = draw_weights(seed, sizes, init)
    spec = Spec(f"custom-{'-'.join(map(str, sizes))}", sizes, onehot, n, n, 0.1, 0.9, 1, seed,
                "onehot" if onehot else input_kind, target_p, init)
    return Workload(spec, sizes, n, x, act, t, w)


def dense_from_active(active: np.ndarray, n0: int) -> np.ndarray:
    """0/1 float32 matrix with ones at the active indices of each row."""
    n = active.shape[0]
    x = np.zeros((n, n0), dtype=np.float32)
    if n:
        rows = np.repeat(np.arange(n), active.shape[1])
        x[rows, active.reshape(-1)] = 1.0
    return x
