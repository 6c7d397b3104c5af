"""ctypes declarations of the C ABI (include/ot_status.h, reservoir.h, surrogate.h).

Argument marshalling only.  Loading fails loudly when the library has not been
built: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libonline_train.so")

OT_OK = 0
OT_NOT_READY = 1
OT_EMPTY = 3
OT_E_INVAL = -1
OT_E_NOMEM = -2
OT_E_HIP = -3
OT_E_CLOSED = -4
OT_E_STATE = -5
OT_FP32 = 0
OT_BF16 = 1
OT_SURROGATE_KEEP_GRADS = 1
OT_POLICY_RESERVOIR = 0
OT_POLICY_FIFO = 1
OT_POLICY_FIRO = 2
OT_PREDICT_NOALLOC_SCRATCH_BYTES = 64 << 20

SURROGATE_PHASES = ("fwd_hidden", "fwd_output", "loss", "wgrad_output", "igrad_output", "igrad_reduce",
                    "bwd_hidden", "adam", "wgrad_reduce")
RESERVOIR_PHASES = ("put_assign", "put_copy", "select", "gather")


class ReservoirStats(C.Structure):
    _fields_ = [(name, C.c_int64) for name in (
        "capacity", "threshold", "n", "unseen", "seen", "total_put", "total_evicted",
        "total_deleted", "total_draws", "next_ticket", "next_sample_id")] + [
        ("reception_over", C.c_int32), ("hist_len", C.c_int32), ("policy", C.c_int32), ("reserved", C.c_int32)]


vp = C.c_void_p
i64 = C.c_int64
i32 = C.c_int32
u64 = C.c_uint64
u32 = C.c_uint32
f32 = C.c_float

SIGNATURES = {
    "ot_last_error": (C.c_char_p, []),
    "ot_version": (C.c_char_p, []),
    "reservoir_create": (C.c_int, [C.POINTER(vp), i64, i64, i64, i64, u64, i32, vp]),
    "reservoir_put": (C.c_int, [vp, vp, i64, vp, i64, i64, vp, vp, C.POINTER(u64)]),
    "reservoir_sample_batch": (C.c_int, [vp, i64, vp, vp, vp, i64, vp, i64, C.POINTER(i64), C.POINTER(u64)]),
    "reservoir_end_reception": (C.c_int, [vp]),
    "reservoir_stats": (C.c_int, [vp, C.POINTER(ReservoirStats)]),
    "reservoir_slab": (C.c_int, [vp, vp, vp, vp, vp]),
    "reservoir_read_meta": (C.c_int, [vp, vp, vp, vp]),
    "reservoir_read_rows": (C.c_int, [vp, vp, i64, vp, vp]),
    "reservoir_timing_begin": (C.c_int, [vp, u32, i64]),
    "reservoir_timing_end": (C.c_int, [vp, vp, vp]),
    "reservoir_destroy": (C.c_int, [vp]),
    "surrogate_create": (C.c_int, [C.POINTER(vp), C.POINTER(i64), i32, i32, f32, f32, f32, f32, u64, i64, u32]),
    "surrogate_set_params": (C.c_int, [vp, i32, vp, vp]),
    "surrogate_get_params": (C.c_int, [vp, i32, vp, vp]),
    "surrogate_get_grads": (C.c_int, [vp, i32, vp, vp]),
    "surrogate_eval_loss": (C.c_int, [vp, vp, i64, vp, i64, i64, vp, vp]),
    "surrogate_checkpoint_size": (C.c_int, [vp, C.POINTER(i64)]),
    "surrogate_checkpoint": (C.c_int, [vp, vp, i64]),
    "surrogate_restore": (C.c_int, [vp, vp, i64]),
    "reservoir_checkpoint_size": (C.c_int, [vp, C.POINTER(i64)]),
    "reservoir_checkpoint": (C.c_int, [vp, vp, i64]),
    "reservoir_restore": (C.c_int, [vp, vp, i64]),
    "surrogate_get_adam_state": (C.c_int, [vp, i32, vp, vp, vp, vp, C.POINTER(i64)]),
    "surrogate_set_lr": (C.c_int, [vp, f32]),
    "surrogate_set_device_step": (C.c_int, [vp, i32]),
    "surrogate_train_step": (C.c_int, [vp, vp, i64, vp, i64, i64, vp, vp]),
    "surrogate_train_step_rows": (C.c_int, [vp, vp, i64, vp, i64, vp, i64, i64, vp, vp, vp]),
    "surrogate_predict": (C.c_int, [vp, vp, i64, i64, vp, i64, vp]),
    "surrogate_predict_noalloc": (C.c_int, [vp, vp, i64, i64, vp, i64, vp]),
    "surrogate_timing_begin": (C.c_int, [vp, u32, i64]),
    "surrogate_timing_end": (C.c_int, [vp, vp, vp]),
    "surrogate_destroy": (C.c_int, [vp]),
}

_lib = None


def load(path: str = LIB_PATH):
    """Load the shared library and declare every entry point (cached)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"HIP library {path} is missing: build it with paper_2309_16743_amd.build.build() "
            "(there is no CPU fallback)")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def last_error() -> str:
    return load().ot_last_error().decode()


class OTError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed with status {status}: {last_error()}")
        self.status = status


def check(fn: str, status: int) -> int:
    if status < 0:
        raise OTError(fn, status)
    return status
