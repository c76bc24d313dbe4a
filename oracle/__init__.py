"""Python handle on the CPU oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package.  It loads ``liboracle.so`` (built from ``bp_oracle.cpp`` by
``oracle/build.py``) and marshals numpy arrays; all arithmetic is in the C++
file.  It shares nothing with the HIP library.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)


def load():
    """Loads liboracle.so, building it first if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build
        build.build()
    lib = ctypes.CDLL(LIB_PATH)
    vp = ctypes.c_void_p
    sig = {
        "orc_create": (vp, [_i32p, ctypes.c_int32, ctypes.c_int32]),
        "orc_destroy": (None, [vp]),
        "orc_num_weights": (ctypes.c_int64, [vp]),
        "orc_set_threads": (None, [ctypes.c_int32]),
        "orc_get_threads": (ctypes.c_int32, []),
        "orc_set_weights": (ctypes.c_int, [vp, _f64p, ctypes.c_int64]),
        "orc_get_weights": (ctypes.c_int, [vp, _f64p, ctypes.c_int64]),
        "orc_set_momentum": (ctypes.c_int, [vp, _f64p, ctypes.c_int64]),
        "orc_get_momentum": (ctypes.c_int, [vp, _f64p, ctypes.c_int64]),
        "orc_forward": (ctypes.c_int, [vp, _f32p, ctypes.c_int64, _f64p]),
        "orc_forward_onehot": (ctypes.c_int, [vp, _i32p, ctypes.c_int32, ctypes.c_int64, _f64p]),
        "orc_gradient": (ctypes.c_int, [vp, _f32p, _f32p, ctypes.c_int64, _f64p, _f64p]),
        "orc_gradient_onehot": (ctypes.c_int, [vp, _i32p, ctypes.c_int32, _f32p, ctypes.c_int64, _f64p, _f64p]),
        "orc_batch_state": (ctypes.c_int, [vp, _f32p, _f32p, ctypes.c_int64, _f64p, _f64p]),
        "orc_train_epoch": (ctypes.c_int, [vp, _f32p, _f32p, ctypes.c_int64, ctypes.c_int32,
                                           ctypes.c_double, ctypes.c_double, _f64p, _f64p]),
        "orc_train_epoch_onehot": (ctypes.c_int, [vp, _i32p, ctypes.c_int32, _f32p, ctypes.c_int64,
                                                  ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                                  _f64p, _f64p]),
        "orc_set_sigmoid": (ctypes.c_int, [vp, ctypes.c_int32]),
        "orc_eval_sigmoid": (ctypes.c_int, [vp, _f64p, ctypes.c_int64, _f64p]),
        "orc_set_fault_limit": (ctypes.c_int, [vp, ctypes.c_double]),
        "orc_fault_count": (ctypes.c_int64, [vp]),
        "orc_checkpoint_save": (ctypes.c_int, [vp]),
        "orc_checkpoint_restore": (ctypes.c_int, [vp]),
        "orc_guard_config": (ctypes.c_int, [vp, ctypes.c_int32, ctypes.c_double]),
        "orc_guard_epoch": (ctypes.c_int, [vp, ctypes.c_double]),
        "orc_set_context": (ctypes.c_int, [vp, ctypes.c_int32, _i32p, _i32p]),
        "orc_train_sequences": (ctypes.c_int, [vp, _f32p, _f32p, _f32p, _f32p, ctypes.c_int64, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_double, ctypes.c_double, _f64p, _f64p]),
        "orc_forward_sequences": (ctypes.c_int, [vp, _f32p, _f32p, ctypes.c_int64, ctypes.c_int32, _f64p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _p(a: Optional[np.ndarray], ptype):
    if a is None:
        return ctypes.cast(None, ptype)
    return a.ctypes.data_as(ptype)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def set_threads(n: int) -> None:
    load().orc_set_threads(int(n))


def get_threads() -> int:
    return int(load().orc_get_threads())


class OracleError(RuntimeError):
    pass


class OracleNet:
    """A fully connected sigmoid net held by the oracle.

    ``storage`` is 64 (the plain definition, double everywhere) or 32 (float
    storage at the points a float32 implementation rounds, double sums).
    Weights use the flat layout: for each layer, (n_l + 1) x n_{l+1}
    row-major, input-major, last row = bias ("true unit").
    """

    def __init__(self, sizes: Sequence[int], storage: int = 64):
        lib = load()
        self.sizes = tuple(int(v) for v in sizes)
        arr = (ctypes.c_int32 * len(self.sizes))(*self.sizes)
        self._h = lib.orc_create(arr, len(self.sizes), int(storage))
        if not self._h:
            raise OracleError(f"bad net sizes {self.sizes} or storage {storage}")
        self.storage = storage
        self.n_weights = int(lib.orc_num_weights(self._h))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h and _lib is not None:
            _lib.orc_destroy(h)
            self._h = None

    def _chk(self, rc: int, what: str):
        if rc != 0:
            raise OracleError(f"{what} rejected its arguments")

    # state -------------------------------------------------------------
    def set_weights(self, w) -> None:
        w = np.ascontiguousarray(w, dtype=np.float64).reshape(-1)
        self._chk(_lib.orc_set_weights(self._h, _p(w, _f64p), w.size), "set_weights")

    def get_weights(self) -> np.ndarray:
        w = np.empty(self.n_weights, np.float64)
        self._chk(_lib.orc_get_weights(self._h, _p(w, _f64p), w.size), "get_weights")
        return w

    def set_momentum(self, v) -> None:
        v = np.ascontiguousarray(v, dtype=np.float64).reshape(-1)
        self._chk(_lib.orc_set_momentum(self._h, _p(v, _f64p), v.size), "set_momentum")

    def get_momentum(self) -> np.ndarray:
        v = np.empty(self.n_weights, np.float64)
        self._chk(_lib.orc_get_momentum(self._h, _p(v, _f64p), v.size), "get_momentum")
        return v

    def layers(self, flat: np.ndarray):
        """Splits a flat weight-shaped array into per-layer (n_l + 1) x n_{l+1} views."""
        out, o = [], 0
        for l in range(len(self.sizes) - 1):
            r, c = self.sizes[l] + 1, self.sizes[l + 1]
            out.append(flat[o:o + r * c].reshape(r, c))
            o += r * c
        return out

    # options -------------------------------------------------------------
    SIGMOID_EXACT, SIGMOID_TABLE = 0, 1

    def set_sigmoid(self, mode: int) -> None:
        """0: exact logistic; 1: the 256-entry interpolated table on [-15, 15] (section 4.3)."""
        self._chk(_lib.orc_set_sigmoid(self._h, int(mode)), "set_sigmoid")

    def eval_sigmoid(self, z) -> np.ndarray:
        """The net's unit nonlinearity at each z (rounded to the storage precision)."""
        z = np.ascontiguousarray(z, dtype=np.float64).reshape(-1)
        y = np.empty_like(z)
        self._chk(_lib.orc_eval_sigmoid(self._h, _p(z, _f64p), z.size, _p(y, _f64p)), "eval_sigmoid")
        return y

    def set_fault_limit(self, limit: float) -> None:
        """Range check of the summed changes (section 8): limit > 0 enables, 0 disables; resets the count."""
        self._chk(_lib.orc_set_fault_limit(self._h, float(limit)), "set_fault_limit")

    def fault_count(self) -> int:
        return int(_lib.orc_fault_count(self._h))

    def checkpoint_save(self) -> None:
        self._chk(_lib.orc_checkpoint_save(self._h), "checkpoint_save")

    def checkpoint_restore(self) -> None:
        self._chk(_lib.orc_checkpoint_restore(self._h), "checkpoint_restore")

    def guard_config(self, every: int, jump: float) -> None:
        """Checkpoint now and every `every` accepted epochs; roll back when an epoch's error > jump x the last."""
        self._chk(_lib.orc_guard_config(self._h, int(every), float(jump)), "guard_config")

    def guard_epoch(self, sse: float) -> int:
        """Reports an epoch's error; returns 1 if the net was rolled back to its checkpoint, else 0."""
        rc = int(_lib.orc_guard_epoch(self._h, float(sse)))
        if rc < 0:
            raise OracleError("guard_epoch: guard not configured")
        return rc

    # recurrence (Elman nets, section 10.5) ---------------------------------
    def set_context(self, from_layer, from_unit) -> None:
        """Context unit c (input unit n_0 - n_ctx + c) copies unit from_unit[c] of hidden layer from_layer[c]."""
        fl, fu = _i32(from_layer).reshape(-1), _i32(from_unit).reshape(-1)
        if fl.size != fu.size:
            raise OracleError("set_context: from_layer and from_unit differ in length")
        self._chk(_lib.orc_set_context(self._h, fl.size, _p(fl, _i32p), _p(fu, _i32p)), "set_context")

    def train_sequences(self, x, t, cont, mask, steps_per_update: int, lr: float, momentum: float,
                        per_window: bool = False):
        """Elman training over [n_steps][n_streams] patterns; returns the summed squared error."""
        x, t, cont, mask = _f32(x), _f32(t), _f32(cont), _f32(mask)
        T, S = cont.shape
        nw = (T + steps_per_update - 1) // steps_per_update if steps_per_update > 0 else 0
        wsse = np.zeros(max(nw, 1), np.float64)
        sse = ctypes.c_double(0.0)
        rc = _lib.orc_train_sequences(self._h, _p(x, _f32p), _p(t, _f32p), _p(cont, _f32p), _p(mask, _f32p), T, S,
                                      int(steps_per_update), float(lr), float(momentum), ctypes.byref(sse),
                                      _p(wsse, _f64p))
        self._chk(rc, "train_sequences")
        return (sse.value, wsse[:nw]) if per_window else sse.value

    def forward_sequences(self, x, cont) -> np.ndarray:
        """Outputs [n_steps][n_streams][n_L] of the sequences at the current weights."""
        x, cont = _f32(x), _f32(cont)
        T, S = cont.shape
        y = np.empty((T, S, self.sizes[-1]), np.float64)
        self._chk(_lib.orc_forward_sequences(self._h, _p(x, _f32p), _p(cont, _f32p), T, S, _p(y, _f64p)),
                  "forward_sequences")
        return y

    # method --------------------------------------------------------------
    def forward(self, x=None, active=None) -> np.ndarray:
        nL = self.sizes[-1]
        if active is not None:
            a = _i32(active)
            y = np.empty((a.shape[0], nL), np.float64)
            self._chk(_lib.orc_forward_onehot(self._h, _p(a, _i32p), a.shape[1] if a.ndim == 2 else 0,
                                              a.shape[0], _p(y, _f64p)), "forward_onehot")
            return y
        x = _f32(x)
        y = np.empty((x.shape[0], nL), np.float64)
        self._chk(_lib.orc_forward(self._h, _p(x, _f32p), x.shape[0], _p(y, _f64p)), "forward")
        return y

    def gradient(self, t, x=None, active=None):
        """Summed weight change direction G over all given patterns (no update); returns (G, sse)."""
        t = _f32(t)
        G = np.empty(self.n_weights, np.float64)
        sse = ctypes.c_double(0.0)
        if active is not None:
            a = _i32(active)
            rc = _lib.orc_gradient_onehot(self._h, _p(a, _i32p), a.shape[1], _p(t, _f32p), a.shape[0],
                                          _p(G, _f64p), ctypes.byref(sse))
        else:
            x = _f32(x)
            rc = _lib.orc_gradient(self._h, _p(x, _f32p), _p(t, _f32p), x.shape[0], _p(G, _f64p),
                                   ctypes.byref(sse))
        self._chk(rc, "gradient")
        return G, sse.value

    def batch_state(self, x, t):
        """Activations a_1..a_L and deltas delta_1..delta_L (lists of [n][n_l]) at the current weights."""
        x, t = _f32(x), _f32(t)
        n = x.shape[0]
        tot = n * sum(self.sizes[1:])
        acts = np.empty(tot, np.float64)
        dels = np.empty(tot, np.float64)
        self._chk(_lib.orc_batch_state(self._h, _p(x, _f32p), _p(t, _f32p), n, _p(acts, _f64p),
                                       _p(dels, _f64p)), "batch_state")
        A, D, o = [], [], 0
        for nl in self.sizes[1:]:
            A.append(acts[o:o + n * nl].reshape(n, nl))
            D.append(dels[o:o + n * nl].reshape(n, nl))
            o += n * nl
        return A, D

    def train_epoch(self, t, batch: int, lr: float, momentum: float, x=None, active=None,
                    per_batch: bool = False):
        """One pass over the patterns in order, one pooled update per batch; returns the summed squared error."""
        t = _f32(t)
        n = t.shape[0]
        nb = (n + batch - 1) // batch if batch > 0 else 0
        bsse = np.zeros(max(nb, 1), np.float64)
        sse = ctypes.c_double(0.0)
        if active is not None:
            a = _i32(active)
            rc = _lib.orc_train_epoch_onehot(self._h, _p(a, _i32p), a.shape[1] if a.ndim == 2 else 0,
                                             _p(t, _f32p), n, int(batch), float(lr), float(momentum),
                                             ctypes.byref(sse), _p(bsse, _f64p))
        else:
            x = _f32(x)
            rc = _lib.orc_train_epoch(self._h, _p(x, _f32p), _p(t, _f32p), n, int(batch), float(lr),
                                      float(momentum), ctypes.byref(sse), _p(bsse, _f64p))
        self._chk(rc, "train_epoch")
        return (sse.value, bsse[:nb]) if per_batch else sse.value
