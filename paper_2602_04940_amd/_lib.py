"""ctypes binding of include/ts3.h: argument marshalling only.

Every computation happens in libts3.so's HIP kernels.  The library must have
been built (``__graft_entry__.build()``); loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes as ct
import os

from .build import LIB

TS3_OK, TS3_ERR_INVALID_ARG, TS3_ERR_BAD_STATE, TS3_ERR_OUT_OF_MEMORY, TS3_ERR_HIP, TS3_ERR_UNSUPPORTED = range(6)
TS3_FP32, TS3_BF16 = 0, 1
TS3_S_RAW, TS3_D, TS3_S, TS3_S1, TS3_ZP, TS3_T_RAW = range(6)


TS3_ACCUM_FP32, TS3_ACCUM_FP64 = 0, 1


class Desc(ct.Structure):
    _fields_ = [("C", ct.c_int32), ("H", ct.c_int32), ("M", ct.c_int32), ("dh", ct.c_int32),
                ("temperature", ct.c_float), ("eps", ct.c_float), ("io_dtype", ct.c_int32),
                ("accum", ct.c_int32), ("group_span", ct.c_int64), ("max_points", ct.c_int64)]


class Weights(ct.Structure):
    _fields_ = [(n, ct.c_void_p) for n in ("W2", "b2", "W1", "b1", "Wq", "Wk", "Wv", "W3", "b3")]


WEIGHT_NAMES = [n for n, _ in Weights._fields_]


class Grads(ct.Structure):
    _fields_ = [(n, ct.c_void_p) for n in ("dW2", "db2", "dW1", "db1", "dWq", "dWk", "dWv", "dW3", "db3")]


GRAD_NAMES = [n for n, _ in Grads._fields_]

BLOCK_EXTRA_NAMES = ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "Wa", "ba", "Wb", "bb")


class BlockWeights(ct.Structure):
    _fields_ = [("pa", Weights)] + [(n, ct.c_void_p) for n in BLOCK_EXTRA_NAMES]

_P = ct.c_void_p
# name -> (restype, argtypes); must match include/ts3.h
SIGNATURES = {
    "ts3_state_create": (ct.c_int, [ct.POINTER(Desc), ct.POINTER(_P)]),
    "ts3_state_free": (ct.c_int, [_P]),
    "ts3_state_bytes": (ct.c_int, [_P, ct.POINTER(ct.c_int64)]),
    "ts3_state_projected": (ct.c_int, [_P, ct.POINTER(ct.c_int32)]),
    "ts3_state_reset": (ct.c_int, [_P, _P]),
    "ts3_slice_accumulate": (ct.c_int, [_P, ct.POINTER(Weights), _P, ct.c_int64, ct.c_int64, _P]),
    "ts3_slice_finalize": (ct.c_int, [_P, ct.POINTER(Weights), _P]),
    "ts3_token_attention": (ct.c_int, [_P, ct.POINTER(Weights), _P]),
    "ts3_deslice": (ct.c_int, [_P, ct.POINTER(Weights), _P, ct.c_int64, _P, _P]),
    "ts3_layer_forward": (ct.c_int, [_P, ct.POINTER(Weights), _P, ct.c_int64, ct.c_int64, ct.c_int64, _P, _P]),
    "ts3_layer_forward_noalloc": (ct.c_int, [ct.POINTER(Desc), ct.POINTER(Weights), _P, ct.c_int64, ct.c_int64,
                                             ct.c_int64, _P, _P]),
    "ts3_layer_backward": (ct.c_int, [_P, ct.POINTER(Weights), _P, _P, ct.c_int64, ct.c_int64, _P,
                                      ct.POINTER(Grads), _P]),
    "ts3_state_get": (ct.c_int, [_P, ct.c_int32, _P, ct.c_int64, _P]),
    "ts3_state_get_spans": (ct.c_int, [_P, ct.c_int64, ct.c_int64, _P, ct.c_int64, _P]),
    "ts3_state_set": (ct.c_int, [_P, ct.POINTER(Weights), ct.c_int32, _P, ct.c_int64, _P, _P]),
    "ts3_stack_create": (ct.c_int, [ct.POINTER(Desc), ct.c_int32, ct.c_int32, ct.POINTER(_P)]),
    "ts3_stack_free": (ct.c_int, [_P]),
    "ts3_stack_bytes": (ct.c_int, [_P, ct.POINTER(ct.c_int64)]),
    "ts3_stack_layer": (ct.c_int, [_P, ct.c_int32, ct.POINTER(_P)]),
    "ts3_stack_forward": (ct.c_int, [_P, ct.POINTER(BlockWeights), _P, ct.c_int64, ct.c_int64, ct.c_int64, _P]),
    "ts3_stack_decode": (ct.c_int, [_P, ct.POINTER(BlockWeights), _P, ct.c_int64, ct.c_int64, _P]),
    "ts3_stack_feedforward": (ct.c_int, [_P, ct.POINTER(BlockWeights), ct.c_int32, _P, _P, ct.c_int64, _P, _P]),
    "ts3_status_string": (ct.c_char_p, [ct.c_int]),
    "ts3_last_error": (ct.c_char_p, []),
}

_lib = None


class TS3Error(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


def lib() -> ct.CDLL:
    """The loaded library; TS3_LIB may name another build of it (default: in-tree)."""
    global _lib
    if _lib is None:
        path = os.environ.get("TS3_LIB", LIB)
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                               "(the layer has no fallback path)")
        L = ct.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def check(status: int, where: str) -> None:
    if status != TS3_OK:
        L = lib()
        raise TS3Error(status, where, f"{L.ts3_status_string(status).decode()}: {L.ts3_last_error().decode()}")
