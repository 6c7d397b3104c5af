"""MI355X (gfx950) online surrogate training: GPU training reservoir + MLP train step.

Thin Python binding over the C ABI of libonline_train.so (include/*.h).  The
functions below carry the C names and only marshal arguments: torch tensors
supply device pointers and HIP streams; every step of the path runs in the
library's HIP kernels.  Importing this package does not touch the GPU; the
first call loads the library and raises if it was not built.
"""
from __future__ import annotations

import ctypes as C
from typing import Optional

import numpy as np

from . import _abi
from ._abi import (OT_BF16, OT_E_CLOSED, OT_E_INVAL, OT_E_STATE, OT_EMPTY, OT_FP32, OT_NOT_READY, OT_OK,
                   OT_POLICY_FIFO, OT_POLICY_FIRO, OT_POLICY_RESERVOIR, OT_SURROGATE_KEEP_GRADS, OTError,
                   check, last_error, load)

__all__ = [
    "Reservoir", "Surrogate", "reservoir_create", "reservoir_put", "reservoir_sample_batch",
    "reservoir_end_reception", "reservoir_stats", "reservoir_read_meta", "reservoir_read_rows",
    "reservoir_destroy", "surrogate_create", "surrogate_set_params", "surrogate_get_params",
    "surrogate_get_grads", "surrogate_get_adam_state", "surrogate_set_lr", "surrogate_train_step",
    "surrogate_predict", "surrogate_predict_noalloc", "surrogate_eval_loss", "surrogate_checkpoint", "surrogate_restore",
    "reservoir_checkpoint", "reservoir_restore", "surrogate_destroy", "load", "last_error", "OTError",
    "OT_OK", "OT_NOT_READY", "OT_EMPTY", "OT_E_INVAL", "OT_E_CLOSED", "OT_E_STATE", "OT_FP32", "OT_BF16",
    "OT_SURROGATE_KEEP_GRADS", "OT_POLICY_RESERVOIR", "OT_POLICY_FIFO", "OT_POLICY_FIRO",
]


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dev_ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return t.data_ptr()


def _rows(t, what: str):
    """(pointer, leading dimension) of a 2-D fp32 device tensor with unit column stride."""
    if t is None:
        return None, 0
    import torch
    if t.dtype != torch.float32 or t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{what}: expected a 2-D float32 tensor with unit column stride")
    return _dev_ptr(t), t.stride(0) if t.shape[0] > 1 else max(t.stride(0), t.shape[1])


def _checkpoint(handle, kind: str) -> np.ndarray:
    lib = load()
    n = C.c_int64()
    check(f"{kind}_checkpoint_size", getattr(lib, f"{kind}_checkpoint_size")(handle, C.byref(n)))
    buf = np.empty(n.value, np.uint8)
    check(f"{kind}_checkpoint", getattr(lib, f"{kind}_checkpoint")(handle, buf.ctypes.data, buf.nbytes))
    return buf


class Reservoir:
    """Handle of one GPU training reservoir (include/reservoir.h)."""

    def __init__(self, capacity: int, threshold: int, x_dim: int, u_dim: int, seed: int,
                 order_stream=None, policy: int = OT_POLICY_RESERVOIR):
        lib = load()
        h = C.c_void_p()
        st = None if order_stream is None else _stream_handle(order_stream)
        check("reservoir_create", lib.reservoir_create(C.byref(h), capacity, threshold, x_dim, u_dim, seed, policy,
                                                       st))
        self.policy = policy
        self._h = h
        self.capacity, self.threshold, self.x_dim, self.u_dim = capacity, threshold, x_dim, u_dim

    @property
    def handle(self):
        return self._h

    def put(self, x, u, stream=None, accepted=None) -> int:
        """Offer the rows of u (and x); returns the ticket.  accepted: device int64[1]."""
        xp, ldx = _rows(x, "x")
        up, ldu = _rows(u, "u")
        k = 0 if u is None else u.shape[0]
        t = C.c_uint64()
        check("reservoir_put", load().reservoir_put(self._h, xp, ldx, up, ldu, k, _stream_handle(stream),
                                                    _dev_ptr(accepted), C.byref(t)))
        return t.value

    def sample_batch(self, b: int, slots, x_out=None, u_out=None, stream=None):
        """Returns (status, rows drawn, ticket or None)."""
        xp, ldx = _rows(x_out, "x_out")
        up, ldu = _rows(u_out, "u_out")
        cnt = C.c_int64()
        t = C.c_uint64()
        st = check("reservoir_sample_batch",
                   load().reservoir_sample_batch(self._h, b, _stream_handle(stream), _dev_ptr(slots), xp, ldx,
                                                 up, ldu, C.byref(cnt), C.byref(t)))
        return st, cnt.value, (t.value if st == OT_OK else None)

    def end_reception(self) -> None:
        check("reservoir_end_reception", load().reservoir_end_reception(self._h))

    def slab(self):
        """(x address, ldx, u address, ldu) of the slabs: slot k's rows start at
        x + 4 ldx k and u + 4 ldu k (bytes)."""
        x, u = C.c_void_p(), C.c_void_p()
        ldx, ldu = C.c_int64(), C.c_int64()
        check("reservoir_slab", load().reservoir_slab(self._h, C.byref(x), C.byref(ldx), C.byref(u), C.byref(ldu)))
        return x.value, ldx.value, u.value, ldu.value

    def stats(self) -> dict:
        s = _abi.ReservoirStats()
        check("reservoir_stats", load().reservoir_stats(self._h, C.byref(s)))
        return {name: getattr(s, name) for name, _ in s._fields_}

    def read_meta(self):
        seen = np.empty(self.capacity, np.int32)
        ids = np.empty(self.capacity, np.int64)
        hist = np.empty(self.stats()["hist_len"], np.int64)
        check("reservoir_read_meta", load().reservoir_read_meta(self._h, seen.ctypes.data, ids.ctypes.data,
                                                                 hist.ctypes.data))
        return seen, ids, hist

    def read_rows(self, slots):
        slots = np.ascontiguousarray(slots, dtype=np.int32)
        x = np.empty((len(slots), self.x_dim), np.float32)
        u = np.empty((len(slots), self.u_dim), np.float32)
        check("reservoir_read_rows", load().reservoir_read_rows(self._h, slots.ctypes.data, len(slots),
                                                                 x.ctypes.data, u.ctypes.data))
        return x, u

    def checkpoint(self) -> np.ndarray:
        """Synchronous snapshot of the whole reservoir state as a host byte array."""
        return _checkpoint(self._h, "reservoir")

    def restore(self, blob: np.ndarray) -> None:
        b = np.ascontiguousarray(blob, dtype=np.uint8)
        check("reservoir_restore", load().reservoir_restore(self._h, b.ctypes.data, b.nbytes))

    def timing_begin(self, phases, max_calls: int) -> None:
        mask = sum(1 << _abi.RESERVOIR_PHASES.index(p) for p in phases)
        check("reservoir_timing_begin", load().reservoir_timing_begin(self._h, mask, max_calls))

    def timing_end(self) -> dict:
        """{phase: (total ms, calls)} for the phases being timed."""
        n = len(_abi.RESERVOIR_PHASES)
        ms = np.zeros(n, np.float64)
        cnt = np.zeros(n, np.int64)
        check("reservoir_timing_end", load().reservoir_timing_end(self._h, ms.ctypes.data, cnt.ctypes.data))
        return {p: (float(ms[i]), int(cnt[i])) for i, p in enumerate(_abi.RESERVOIR_PHASES) if cnt[i]}

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            check("reservoir_destroy", load().reservoir_destroy(self._h))
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Surrogate:
    """Handle of one MLP surrogate with Adam state (include/surrogate.h)."""

    def __init__(self, widths, precision: int = OT_FP32, lr: float = 1e-3, beta1: float = 0.9,
                 beta2: float = 0.999, eps: float = 1e-8, seed: int = 0, max_batch: int = 1024, flags: int = 0):
        lib = load()
        self.widths = tuple(int(w) for w in widths)
        arr = (C.c_int64 * len(self.widths))(*self.widths)
        h = C.c_void_p()
        check("surrogate_create", lib.surrogate_create(C.byref(h), arr, len(self.widths), precision, lr, beta1,
                                                       beta2, eps, seed, max_batch, flags))
        self._h = h
        self.precision = precision

    @property
    def handle(self):
        return self._h

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    def _layer_arrays(self, layer):
        return (np.empty((self.widths[layer + 1], self.widths[layer]), np.float32),
                np.empty(self.widths[layer + 1], np.float32))

    def set_params(self, layer: int, W=None, b=None) -> None:
        Wc = None if W is None else np.ascontiguousarray(W, dtype=np.float32)
        bc = None if b is None else np.ascontiguousarray(b, dtype=np.float32)
        if Wc is not None:
            assert Wc.shape == (self.widths[layer + 1], self.widths[layer])
        check("surrogate_set_params", load().surrogate_set_params(
            self._h, layer, None if Wc is None else Wc.ctypes.data, None if bc is None else bc.ctypes.data))

    def get_params(self, layer: int):
        W, b = self._layer_arrays(layer)
        check("surrogate_get_params", load().surrogate_get_params(self._h, layer, W.ctypes.data, b.ctypes.data))
        return W, b

    def get_grads(self, layer: int, weights: bool = True):
        """(dW, db) of the last step; dW is None when weights=False (the output
        layer's dW is not stored when its Adam update is fused)."""
        W, b = self._layer_arrays(layer)
        check("surrogate_get_grads", load().surrogate_get_grads(self._h, layer, W.ctypes.data if weights else None,
                                                                b.ctypes.data))
        return (W if weights else None), b

    def get_adam_state(self, layer: int):
        mW, mb = self._layer_arrays(layer)
        vW, vb = self._layer_arrays(layer)
        t = C.c_int64()
        check("surrogate_get_adam_state", load().surrogate_get_adam_state(
            self._h, layer, mW.ctypes.data, mb.ctypes.data, vW.ctypes.data, vb.ctypes.data, C.byref(t)))
        return (mW, mb), (vW, vb), t.value

    def set_lr(self, lr: float) -> None:
        check("surrogate_set_lr", load().surrogate_set_lr(self._h, lr))

    def set_device_step(self, enable: bool) -> None:
        """Adam's step counter in device memory (include/surrogate.h), so that a
        captured train step can be replayed."""
        check("surrogate_set_device_step", load().surrogate_set_device_step(self._h, 1 if enable else 0))

    def train_step(self, x, u, stream=None, loss=None) -> None:
        xp, ldx = _rows(x, "x")
        up, ldu = _rows(u, "u")
        check("surrogate_train_step", load().surrogate_train_step(
            self._h, xp, ldx, up, ldu, u.shape[0], _stream_handle(stream), _dev_ptr(loss)))

    def train_step_rows(self, x, u_addr: int, ldu: int, rows, n_rows: int, stream=None, loss=None,
                        targets_read=None) -> None:
        """Train step whose target row j is the fp32 row at device address
        u_addr + 4 ldu rows[j] (rows: int32 device tensor of x's row count,
        each in [0, n_rows)); targets_read: torch.cuda.Event recorded once the
        targets have been read."""
        import torch
        xp, ldx = _rows(x, "x")
        if rows.dtype != torch.int32 or rows.dim() != 1 or rows.shape[0] != x.shape[0] or not rows.is_contiguous():
            raise ValueError("rows: expected a contiguous int32 tensor with one index per row of x")
        ev = None
        if targets_read is not None:
            targets_read.record(torch.cuda.current_stream() if stream is None else stream)   # create the event
            ev = targets_read.cuda_event
        check("surrogate_train_step_rows", load().surrogate_train_step_rows(
            self._h, xp, ldx, u_addr, ldu, _dev_ptr(rows), n_rows, x.shape[0], _stream_handle(stream),
            _dev_ptr(loss), ev))

    def predict(self, x, y, stream=None) -> None:
        xp, ldx = _rows(x, "x")
        yp, ldy = _rows(y, "y")
        check("surrogate_predict", load().surrogate_predict(self._h, xp, ldx, x.shape[0], yp, ldy,
                                                            _stream_handle(stream)))

    def predict_noalloc(self, x, y, stream=None) -> None:
        """predict() through the entry point that allocates nothing (its
        workspace is the library's per-device scratch; see include/surrogate.h)."""
        xp, ldx = _rows(x, "x")
        yp, ldy = _rows(y, "y")
        check("surrogate_predict_noalloc", load().surrogate_predict_noalloc(self._h, xp, ldx, x.shape[0], yp, ldy,
                                                                            _stream_handle(stream)))

    def checkpoint(self) -> np.ndarray:
        """Synchronous snapshot of parameters, Adam moments and step counter."""
        return _checkpoint(self._h, "surrogate")

    def restore(self, blob: np.ndarray) -> None:
        b = np.ascontiguousarray(blob, dtype=np.uint8)
        check("surrogate_restore", load().surrogate_restore(self._h, b.ctypes.data, b.nbytes))

    def eval_loss(self, x, u, loss, stream=None) -> None:
        """Validation MSE of the current surrogate on rows x -> u into the device scalar `loss`."""
        xp, ldx = _rows(x, "x")
        up, ldu = _rows(u, "u")
        check("surrogate_eval_loss", load().surrogate_eval_loss(self._h, xp, ldx, up, ldu, x.shape[0],
                                                                _stream_handle(stream), _dev_ptr(loss)))

    def timing_begin(self, phases, max_steps: int) -> None:
        mask = sum(1 << _abi.SURROGATE_PHASES.index(p) for p in phases)
        check("surrogate_timing_begin", load().surrogate_timing_begin(self._h, mask, max_steps))

    def timing_end(self) -> dict:
        """{phase: (total ms, steps)} for the phases being timed."""
        n = len(_abi.SURROGATE_PHASES)
        ms = np.zeros(n, np.float64)
        cnt = np.zeros(n, np.int64)
        check("surrogate_timing_end", load().surrogate_timing_end(self._h, ms.ctypes.data, cnt.ctypes.data))
        return {p: (float(ms[i]), int(cnt[i])) for i, p in enumerate(_abi.SURROGATE_PHASES) if cnt[i]}

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            check("surrogate_destroy", load().surrogate_destroy(self._h))
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---- C-named entry points (argument marshalling only) ----------------------------
def reservoir_create(capacity, threshold, x_dim, u_dim, seed, policy=OT_POLICY_RESERVOIR,
                     order_stream=None) -> Reservoir:
    return Reservoir(capacity, threshold, x_dim, u_dim, seed, order_stream, policy)


def reservoir_put(r: Reservoir, x, u, stream=None, accepted=None) -> int:
    return r.put(x, u, stream, accepted)


def reservoir_sample_batch(r: Reservoir, b, slots, x_out=None, u_out=None, stream=None):
    return r.sample_batch(b, slots, x_out, u_out, stream)


def reservoir_end_reception(r: Reservoir) -> None:
    r.end_reception()


def reservoir_stats(r: Reservoir) -> dict:
    return r.stats()


def reservoir_read_meta(r: Reservoir):
    return r.read_meta()


def reservoir_read_rows(r: Reservoir, slots):
    return r.read_rows(slots)


def reservoir_destroy(r: Reservoir) -> None:
    r.close()


def surrogate_create(widths, precision=OT_FP32, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, seed=0,
                     max_batch=1024, flags=0) -> Surrogate:
    return Surrogate(widths, precision, lr, beta1, beta2, eps, seed, max_batch, flags)


def surrogate_set_params(s: Surrogate, layer, W=None, b=None) -> None:
    s.set_params(layer, W, b)


def surrogate_get_params(s: Surrogate, layer):
    return s.get_params(layer)


def reservoir_checkpoint(r: Reservoir) -> np.ndarray:
    return r.checkpoint()


def reservoir_restore(r: Reservoir, blob) -> None:
    r.restore(blob)


def surrogate_checkpoint(s: Surrogate) -> np.ndarray:
    return s.checkpoint()


def surrogate_restore(s: Surrogate, blob) -> None:
    s.restore(blob)


def surrogate_eval_loss(s: Surrogate, x, u, loss, stream=None):
    return s.eval_loss(x, u, loss, stream)


def surrogate_get_grads(s: Surrogate, layer):
    return s.get_grads(layer)


def surrogate_get_adam_state(s: Surrogate, layer):
    return s.get_adam_state(layer)


def surrogate_set_lr(s: Surrogate, lr) -> None:
    s.set_lr(lr)


def surrogate_train_step(s: Surrogate, x, u, stream=None, loss=None) -> None:
    s.train_step(x, u, stream, loss)


def surrogate_predict(s: Surrogate, x, y, stream=None) -> None:
    s.predict(x, y, stream)


def surrogate_predict_noalloc(s: Surrogate, x, y, stream=None) -> None:
    s.predict_noalloc(x, y, stream)


def surrogate_destroy(s: Surrogate) -> None:
    s.close()
