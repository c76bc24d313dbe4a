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


# ---------------------------------------------------------------------------
# Sequences for Elman nets (section 10.5).  The paper's speech data is not
# available; these synthetic sequences stand in with its structure: frames
# of features, a class per frame, sequences of mixed length packed into
# parallel streams (one stream per processor in the paper), the padding
# after a stream's last whole sequence marked by a zero mask flag.
#
# Recipe (streams 3, 4, 5 of the seed: sequence layout, frames, weights):
#   * stream s is filled with sequences of length integers(len_min,
#     len_max + 1) while the next one fits in n_steps; continuation flag 0 at
#     each sequence start and 1 inside; steps after the last sequence get
#     continuation 0 and mask 0, other steps mask 1;
#   * a sequence is a run of segments of integers(3, 11) frames; each
#     segment has a class uniform over the n_out classes; a frame's features
#     are that class's embedding (standard normal, n_out x n_ext, one per
#     workload) plus 0.5 standard normal noise;
#   * targets: 0.9 for the frame's class, 0.1 for the others (padding frames
#     draw a class too; their mask is 0);
#   * weights uniform(-1/sqrt(fan_in), 1/sqrt(fan_in)) like the dense nets;
#   * the context (n_ctx units, the last inputs) copies the first n_ctx
#     units of hidden layer 1.

@dataclasses.dataclass(frozen=True)
class SeqSpec:
    name: str
    n_ext: int              # external inputs per frame
    hidden: tuple           # hidden layer sizes
    n_out: int              # classes = output units
    n_ctx: int              # context units (copies of hidden layer 1)
    n_streams: int
    n_steps: int
    steps_per_update: int
    len_min: int
    len_max: int
    lr: float
    momentum: float
    epochs: int
    seed: int
    note: str = ""

    @property
    def sizes(self) -> tuple:
        return (self.n_ext + self.n_ctx,) + tuple(self.hidden) + (self.n_out,)


SEQ_SPECS = {
    s.name: s
    for s in [
        SeqSpec("elman-64+256-256-64", 64, (256,), 64, 256, 1024, 128, 8, 16, 64, 5e-6, 0.9, 1, 6,
                "Elman net, 1024 parallel streams of 16-64-frame sequences, an update every 8 steps"),
        SeqSpec("elman-20+48-48-12", 20, (48,), 12, 48, 200, 37, 5, 4, 12, 5e-4, 0.9, 3, 7,
                "small Elman net with a ragged stream count and a short last window"),
    ]
}


@dataclasses.dataclass
class SeqWorkload:
    spec: SeqSpec
    inputs: np.ndarray      # float32 [n_steps][n_streams][n_ext]
    targets: np.ndarray     # float32 [n_steps][n_streams][n_out]
    cont: np.ndarray        # float32 [n_steps][n_streams]: 1 continues a sequence, 0 starts one
    mask: np.ndarray        # float32 [n_steps][n_streams]: 0 on the padding after a stream's last sequence
    weights: np.ndarray     # float32 flat, C-ABI layout
    ctx_layer: np.ndarray   # int32 [n_ctx]
    ctx_unit: np.ndarray    # int32 [n_ctx]

    @property
    def sizes(self) -> tuple:
        return self.spec.sizes

    @property
    def lr(self) -> float:
        return float(np.float32(self.spec.lr))

    @property
    def momentum(self) -> float:
        return float(np.float32(self.spec.momentum))

    @property
    def n_patterns(self) -> int:
        return self.spec.n_steps * self.spec.n_streams


def make_sequences(spec) -> SeqWorkload:
    """Builds a sequence workload from a SeqSpec or the name of one."""
    s = SEQ_SPECS[spec] if isinstance(spec, str) else spec
    T, S = s.n_steps, s.n_streams
    g_lay, g_frm = _rng(s.seed, 3), _rng(s.seed, 4)
    cont = np.zeros((T, S), np.float32)
    mask = np.zeros((T, S), np.float32)
    cls = np.zeros((T, S), np.int64)
    for st in range(S):
        pos = 0
        while True:
            n = int(g_lay.integers(s.len_min, s.len_max + 1))
            if pos + n > T:
                break
            cont[pos + 1:pos + n, st] = 1.0
            mask[pos:pos + n, st] = 1.0
            pos += n
        # classes in segments over the whole stream (padding included)
        t0 = 0
        while t0 < T:
            m = int(g_lay.integers(3, 11))
            cls[t0:t0 + m, st] = g_lay.integers(0, s.n_out)
            t0 += m
    emb = g_frm.standard_normal((s.n_out, s.n_ext))
    x = np.empty((T, S, s.n_ext), np.float32)
    for t in range(T):
        x[t] = emb[cls[t]] + 0.5 * g_frm.standard_normal((S, s.n_ext))
    tg = np.full((T, S, s.n_out), 0.1, np.float32)
    np.put_along_axis(tg, cls[:, :, None], np.float32(0.9), axis=2)
    w = draw_weights(s.seed, s.sizes, "fanin")
    ctx_layer = np.ones(s.n_ctx, np.int32)
    ctx_unit = np.arange(s.n_ctx, dtype=np.int32)
    return SeqWorkload(s, x, tg, cont, mask, w, ctx_layer, ctx_unit)
