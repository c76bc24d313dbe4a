"""Thin ctypes binding of libbp.so (include/bp.h).

Argument marshalling only: every step of the method runs in the library's
HIP kernels.  The module-level functions carry the C names; ``Net`` wraps a
handle for convenience.  Device buffers are torch tensors on a ROCm device,
passed by pointer; torch supplies device memory and the stream, nothing else.

torch is imported before the library is loaded so that the library binds to
the HIP runtime torch already has in the process (one runtime per process).
If libbp.so has not been built this module raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch  # noqa: F401  (must precede loading libbp.so, see above)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbp.so")

BP_OK, BP_EINVAL, BP_ENOMEM, BP_EDEVICE = 0, -1, -2, -3
EXPORTS = ("bp_create", "bp_destroy", "bp_set_stream", "bp_num_weights", "bp_set_weights", "bp_get_weights",
           "bp_set_momentum", "bp_get_momentum", "bp_train_batches", "bp_train_batches_noalloc",
           "bp_train_batches_onehot", "bp_forward",
           "bp_forward_onehot", "bp_set_context", "bp_train_sequences", "bp_forward_sequences", "bp_set_sigmoid", "bp_set_fault_limit", "bp_get_fault_count",
           "bp_checkpoint_save", "bp_checkpoint_restore", "bp_guard_config", "bp_guard_epoch", "bp_set_graph_replay", "bp_profile",
           "bp_profile_report", "bp_last_error")
BP_SIGMOID_EXACT, BP_SIGMOID_TABLE = 0, 1
KINDS = ("forward", "output", "backward", "change", "splitk", "bias", "gather", "scatter", "reduce", "fused_fb",
         "fused_update", "output_finish", "seq_in", "seq_pair", "seq_win")

_lib = None
_vp = ctypes.c_void_p
_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)


class BPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


def lib():
    """Loads libbp.so (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run paper_1801_01554_amd/build.py (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    sig = {
        "bp_create": (ctypes.c_int, [_i32p, ctypes.c_int32, ctypes.POINTER(_vp)]),
        "bp_destroy": (None, [_vp]),
        "bp_set_stream": (ctypes.c_int, [_vp, _vp]),
        "bp_num_weights": (ctypes.c_int64, [_vp]),
        "bp_set_weights": (ctypes.c_int, [_vp, _f32p, ctypes.c_int64]),
        "bp_get_weights": (ctypes.c_int, [_vp, _f32p, ctypes.c_int64]),
        "bp_set_momentum": (ctypes.c_int, [_vp, _f32p, ctypes.c_int64]),
        "bp_get_momentum": (ctypes.c_int, [_vp, _f32p, ctypes.c_int64]),
        "bp_train_batches": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                                            ctypes.c_float, _f64p]),
        "bp_train_batches_noalloc": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                                                    ctypes.c_float, _f64p]),
        "bp_train_batches_onehot": (ctypes.c_int, [_vp, _vp, ctypes.c_int32, _vp, ctypes.c_int64, ctypes.c_int32,
                                                   ctypes.c_float, ctypes.c_float, _f64p]),
        "bp_forward": (ctypes.c_int, [_vp, _vp, ctypes.c_int64, _vp]),
        "bp_forward_onehot": (ctypes.c_int, [_vp, _vp, ctypes.c_int32, ctypes.c_int64, _vp]),
        "bp_set_context": (ctypes.c_int, [_vp, ctypes.c_int32, _i32p, _i32p]),
        "bp_train_sequences": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_int32,
                                              ctypes.c_int32, ctypes.c_float, ctypes.c_float, _f64p]),
        "bp_forward_sequences": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int64, ctypes.c_int32, _vp]),
        "bp_set_sigmoid": (ctypes.c_int, [_vp, ctypes.c_int32]),
        "bp_set_fault_limit": (ctypes.c_int, [_vp, ctypes.c_float]),
        "bp_get_fault_count": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_int64)]),
        "bp_checkpoint_save": (ctypes.c_int, [_vp]),
        "bp_checkpoint_restore": (ctypes.c_int, [_vp]),
        "bp_guard_config": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_double]),
        "bp_guard_epoch": (ctypes.c_int, [_vp, ctypes.c_double, ctypes.POINTER(ctypes.c_int32)]),
        "bp_set_graph_replay": (ctypes.c_int, [_vp, ctypes.c_int]),
        "bp_profile": (ctypes.c_int, [_vp, ctypes.c_int]),
        "bp_profile_report": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_int64), _f64p, ctypes.c_int32]),
        "bp_last_error": (ctypes.c_char_p, [_vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


# ---------------------------------------------------------------- C names
def bp_create(layer_sizes: Sequence[int]):
    """Returns (rc, handle)."""
    arr = (ctypes.c_int32 * len(layer_sizes))(*[int(v) for v in layer_sizes])
    h = _vp()
    rc = lib().bp_create(arr, len(layer_sizes), ctypes.byref(h))
    return rc, h


def bp_destroy(h) -> None:
    lib().bp_destroy(h)


def bp_set_stream(h, stream_ptr: int) -> int:
    return lib().bp_set_stream(h, _vp(stream_ptr))


def bp_num_weights(h) -> int:
    return int(lib().bp_num_weights(h))


def bp_set_weights(h, w: np.ndarray) -> int:
    return lib().bp_set_weights(h, w.ctypes.data_as(_f32p), w.size)


def bp_get_weights(h, w: np.ndarray) -> int:
    return lib().bp_get_weights(h, w.ctypes.data_as(_f32p), w.size)


def bp_set_momentum(h, v: np.ndarray) -> int:
    return lib().bp_set_momentum(h, v.ctypes.data_as(_f32p), v.size)


def bp_get_momentum(h, v: np.ndarray) -> int:
    return lib().bp_get_momentum(h, v.ctypes.data_as(_f32p), v.size)


def bp_train_batches(h, inputs_ptr: int, targets_ptr: int, n: int, batch: int, lr: float, momentum: float,
                     sse: Optional[ctypes.c_double]) -> int:
    return lib().bp_train_batches(h, _vp(inputs_ptr), _vp(targets_ptr), n, batch, lr, momentum,
                                  ctypes.byref(sse) if sse is not None else None)


def bp_train_batches_noalloc(h, inputs_ptr: int, targets_ptr: int, n: int, batch: int, lr: float, momentum: float,
                             sse: Optional[ctypes.c_double]) -> int:
    return lib().bp_train_batches_noalloc(h, _vp(inputs_ptr), _vp(targets_ptr), n, batch, lr, momentum,
                                          ctypes.byref(sse) if sse is not None else None)


def bp_train_batches_onehot(h, active_ptr: int, n_active: int, targets_ptr: int, n: int, batch: int, lr: float,
                            momentum: float, sse: Optional[ctypes.c_double]) -> int:
    return lib().bp_train_batches_onehot(h, _vp(active_ptr), n_active, _vp(targets_ptr), n, batch, lr, momentum,
                                         ctypes.byref(sse) if sse is not None else None)


def bp_forward(h, inputs_ptr: int, n: int, outputs_ptr: int) -> int:
    return lib().bp_forward(h, _vp(inputs_ptr), n, _vp(outputs_ptr))


def bp_forward_onehot(h, active_ptr: int, n_active: int, n: int, outputs_ptr: int) -> int:
    return lib().bp_forward_onehot(h, _vp(active_ptr), n_active, n, _vp(outputs_ptr))


def bp_set_context(h, from_layer, from_unit) -> int:
    fl = np.ascontiguousarray(from_layer, dtype=np.int32).reshape(-1)
    fu = np.ascontiguousarray(from_unit, dtype=np.int32).reshape(-1)
    if fl.size != fu.size:
        return BP_EINVAL
    return lib().bp_set_context(h, fl.size, fl.ctypes.data_as(_i32p), fu.ctypes.data_as(_i32p))


def bp_train_sequences(h, inputs_ptr: int, targets_ptr: int, cont_ptr: int, mask_ptr: int, n_steps: int,
                       n_streams: int, steps_per_update: int, lr: float, momentum: float,
                       sse: Optional[ctypes.c_double]) -> int:
    return lib().bp_train_sequences(h, _vp(inputs_ptr), _vp(targets_ptr), _vp(cont_ptr), _vp(mask_ptr), n_steps,
                                    n_streams, steps_per_update, lr, momentum,
                                    ctypes.byref(sse) if sse is not None else None)


def bp_forward_sequences(h, inputs_ptr: int, cont_ptr: int, n_steps: int, n_streams: int, outputs_ptr: int) -> int:
    return lib().bp_forward_sequences(h, _vp(inputs_ptr), _vp(cont_ptr), n_steps, n_streams, _vp(outputs_ptr))


def bp_set_sigmoid(h, mode: int) -> int:
    return lib().bp_set_sigmoid(h, int(mode))


def bp_set_fault_limit(h, limit: float) -> int:
    return lib().bp_set_fault_limit(h, float(limit))


def bp_get_fault_count(h):
    """Returns (rc, count)."""
    c = ctypes.c_int64(0)
    rc = lib().bp_get_fault_count(h, ctypes.byref(c))
    return rc, int(c.value)


def bp_checkpoint_save(h) -> int:
    return lib().bp_checkpoint_save(h)


def bp_checkpoint_restore(h) -> int:
    return lib().bp_checkpoint_restore(h)


def bp_guard_config(h, every: int, jump: float) -> int:
    return lib().bp_guard_config(h, int(every), float(jump))


def bp_guard_epoch(h, sse: float):
    """Returns (rc, rolled_back)."""
    r = ctypes.c_int32(0)
    rc = lib().bp_guard_epoch(h, float(sse), ctypes.byref(r))
    return rc, int(r.value)


def bp_set_graph_replay(h, on: bool) -> int:
    return lib().bp_set_graph_replay(h, 1 if on else 0)


def bp_profile(h, on: bool) -> int:
    return lib().bp_profile(h, 1 if on else 0)


def bp_profile_report(h):
    """Returns (rc, {kind: (launches, ms)})."""
    n = len(KINDS)
    cnt = (ctypes.c_int64 * n)()
    ms = (ctypes.c_double * n)()
    rc = lib().bp_profile_report(h, cnt, ms, n)
    return rc, {k: (int(cnt[i]), float(ms[i])) for i, k in enumerate(KINDS)}


def bp_last_error(h) -> str:
    m = lib().bp_last_error(h)
    return m.decode() if m else ""


# ---------------------------------------------------------------- convenience
def _dev_ptr(t: "torch.Tensor", dtype, shape, what: str) -> int:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{what} must be a torch tensor on a ROCm device")
    if t.dtype != dtype or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what}: need contiguous {dtype} of shape {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")
    return t.data_ptr()


class Net:
    """A net on the current ROCm device, enqueueing on torch's current stream."""

    def __init__(self, sizes: Sequence[int], stream: Optional["torch.cuda.Stream"] = None):
        self.sizes = tuple(int(v) for v in sizes)
        rc, h = bp_create(self.sizes)
        if rc != BP_OK:
            raise BPError(rc, bp_last_error(None))
        self._h = h
        self.n_weights = bp_num_weights(h)
        self.set_stream(stream if stream is not None else torch.cuda.current_stream())

    def _chk(self, rc: int):
        if rc != BP_OK:
            raise BPError(rc, bp_last_error(self._h))

    def close(self):
        if getattr(self, "_h", None):
            bp_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_stream(self, stream: "torch.cuda.Stream"):
        self.stream = stream
        self._chk(bp_set_stream(self._h, stream.cuda_stream))

    def set_weights(self, w) -> None:
        w = np.ascontiguousarray(w, dtype=np.float32).reshape(-1)
        self._chk(bp_set_weights(self._h, w))

    def get_weights(self) -> np.ndarray:
        w = np.empty(self.n_weights, np.float32)
        self._chk(bp_get_weights(self._h, w))
        return w

    def set_momentum(self, v) -> None:
        v = np.ascontiguousarray(v, dtype=np.float32).reshape(-1)
        self._chk(bp_set_momentum(self._h, v))

    def get_momentum(self) -> np.ndarray:
        v = np.empty(self.n_weights, np.float32)
        self._chk(bp_get_momentum(self._h, v))
        return v

    def train_batches(self, targets, batch: int, lr: float, momentum: float, inputs=None, active=None,
                      want_sse: bool = True) -> Optional[float]:
        n = int(targets.shape[0])
        tp = _dev_ptr(targets, torch.float32, (n, self.sizes[-1]), "targets")
        sse = ctypes.c_double(0.0) if want_sse else None
        if active is not None:
            k = int(active.shape[1])
            ap = _dev_ptr(active, torch.int32, (n, k), "active")
            rc = bp_train_batches_onehot(self._h, ap, k, tp, n, int(batch), float(lr), float(momentum), sse)
        else:
            xp = _dev_ptr(inputs, torch.float32, (n, self.sizes[0]), "inputs")
            rc = bp_train_batches(self._h, xp, tp, n, int(batch), float(lr), float(momentum), sse)
        self._chk(rc)
        return sse.value if want_sse else None

    def set_context(self, from_layer, from_unit) -> None:
        self._chk(bp_set_context(self._h, from_layer, from_unit))
        self.n_ctx = int(np.asarray(from_layer).size)

    def train_sequences(self, inputs, targets, cont, mask, steps_per_update: int, lr: float, momentum: float,
                        want_sse: bool = True) -> Optional[float]:
        """inputs [T][S][n_0 - n_ctx], targets [T][S][n_L], cont and mask [T][S]: device float tensors."""
        T, S = int(cont.shape[0]), int(cont.shape[1])
        n_ext = self.sizes[0] - getattr(self, "n_ctx", 0)
        xp = _dev_ptr(inputs, torch.float32, (T, S, n_ext), "inputs")
        tp = _dev_ptr(targets, torch.float32, (T, S, self.sizes[-1]), "targets")
        cp = _dev_ptr(cont, torch.float32, (T, S), "cont")
        mp = _dev_ptr(mask, torch.float32, (T, S), "mask")
        sse = ctypes.c_double(0.0) if want_sse else None
        self._chk(bp_train_sequences(self._h, xp, tp, cp, mp, T, S, int(steps_per_update), float(lr),
                                     float(momentum), sse))
        return sse.value if want_sse else None

    def forward_sequences(self, inputs, cont) -> "torch.Tensor":
        T, S = int(cont.shape[0]), int(cont.shape[1])
        n_ext = self.sizes[0] - getattr(self, "n_ctx", 0)
        xp = _dev_ptr(inputs, torch.float32, (T, S, n_ext), "inputs")
        cp = _dev_ptr(cont, torch.float32, (T, S), "cont")
        out = torch.empty((T, S, self.sizes[-1]), dtype=torch.float32, device=cont.device)
        self._chk(bp_forward_sequences(self._h, xp, cp, T, S, out.data_ptr()))
        return out

    def set_sigmoid(self, mode: int) -> None:
        self._chk(bp_set_sigmoid(self._h, mode))

    def set_fault_limit(self, limit: float) -> None:
        self._chk(bp_set_fault_limit(self._h, limit))

    def fault_count(self) -> int:
        rc, c = bp_get_fault_count(self._h)
        self._chk(rc)
        return c

    def checkpoint_save(self) -> None:
        self._chk(bp_checkpoint_save(self._h))

    def checkpoint_restore(self) -> None:
        self._chk(bp_checkpoint_restore(self._h))

    def guard_config(self, every: int, jump: float) -> None:
        self._chk(bp_guard_config(self._h, every, jump))

    def guard_epoch(self, sse: float) -> int:
        rc, r = bp_guard_epoch(self._h, sse)
        self._chk(rc)
        return r

    def set_graph_replay(self, on: bool) -> None:
        """Replay repeated training calls from a captured HIP graph (default on)."""
        self._chk(bp_set_graph_replay(self._h, on))

    def profile(self, on: bool) -> None:
        self._chk(bp_profile(self._h, on))

    def profile_report(self) -> dict:
        rc, rep = bp_profile_report(self._h)
        self._chk(rc)
        return rep

    def forward(self, inputs=None, active=None) -> "torch.Tensor":
        src = active if active is not None else inputs
        n = int(src.shape[0])
        out = torch.empty((n, self.sizes[-1]), dtype=torch.float32, device=src.device)
        if active is not None:
            k = int(active.shape[1])
            ap = _dev_ptr(active, torch.int32, (n, k), "active")
            rc = bp_forward_onehot(self._h, ap, k, n, out.data_ptr())
        else:
            xp = _dev_ptr(inputs, torch.float32, (n, self.sizes[0]), "inputs")
            rc = bp_forward(self._h, xp, n, out.data_ptr())
        self._chk(rc)
        return out
