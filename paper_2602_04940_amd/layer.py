"""Python face of libts3: one Physics-Attention layer on a torch-allocated mesh.

torch provides device memory and the current stream; each method marshals
pointers into the C ABI (include/ts3.h) and every step runs in the library's
HIP kernels.
"""
from __future__ import annotations

import ctypes as ct
import math

import numpy as np
import torch

from . import _lib as L

_DTYPES = {"fp32": (L.TS3_FP32, torch.float32), "bf16": (L.TS3_BF16, torch.bfloat16)}


def _stream():
    return ct.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ct.c_void_p(t.data_ptr()) if t is not None else ct.c_void_p(0)


class LayerWeights:
    """Device float32 copies of the layer weights (see include/ts3.h for shapes)."""

    def __init__(self, weights: dict, device="cuda"):
        self.t = {}
        for n in L.WEIGHT_NAMES:
            v = weights.get(n)
            if v is None:
                self.t[n] = None
                continue
            v = torch.as_tensor(np.asarray(v, dtype=np.float32)) if not torch.is_tensor(v) else v
            self.t[n] = v.to(device=device, dtype=torch.float32).contiguous()
        self.struct = L.Weights(**{n: (self.t[n].data_ptr() if self.t[n] is not None else None)
                                   for n in L.WEIGHT_NAMES})

    def ref(self):
        return ct.byref(self.struct)


class PhysicsAttention:
    """A layer state: pass 1 accumulation, token-side work, pass 2 decoding."""

    def __init__(self, C, H, M, dh=None, temperature=0.5, dtype="bf16", group_span=32768,
                 max_points=1 << 20, eps=0.0, accum="fp32"):
        self.C, self.H, self.M = C, H, M
        self.dh = C // H if dh is None else dh
        self.dtype_name = dtype
        code, self.torch_dtype = _DTYPES[dtype]
        acc = {"fp32": L.TS3_ACCUM_FP32, "fp64": L.TS3_ACCUM_FP64}[accum]
        self.desc = L.Desc(C=C, H=H, M=M, dh=self.dh, temperature=temperature, eps=eps, io_dtype=code,
                           accum=acc, group_span=group_span, max_points=max_points)
        h = ct.c_void_p()
        L.check(L.lib().ts3_state_create(ct.byref(self.desc), ct.byref(h)), "ts3_state_create")
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            L.check(L.lib().ts3_state_free(self.h), "ts3_state_free")
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # ----------------------------------------------------------- helpers
    def _check_x(self, x, name="x"):
        if not (x.is_cuda and x.dtype == self.torch_dtype and x.is_contiguous() and x.dim() == 2
                and x.shape[1] == self.C):
            raise ValueError(f"{name} must be a contiguous cuda {self.torch_dtype} tensor [n, {self.C}]")

    def bytes(self) -> int:
        b = ct.c_int64()
        L.check(L.lib().ts3_state_bytes(self.h, ct.byref(b)), "ts3_state_bytes")
        return b.value

    def projected(self) -> bool:
        """True when pass 1 sums x_i W1_h per head (rows of dh + 1) instead of x_i."""
        v = ct.c_int32()
        L.check(L.lib().ts3_state_projected(self.h, ct.byref(v)), "ts3_state_projected")
        return bool(v.value)

    # ----------------------------------------------------------- ABI calls
    def reset(self):
        L.check(L.lib().ts3_state_reset(self.h, _stream()), "ts3_state_reset")

    def accumulate(self, w: LayerWeights, x_tile, point_offset: int):
        self._check_x(x_tile, "x_tile")
        L.check(L.lib().ts3_slice_accumulate(self.h, w.ref(), _ptr(x_tile), x_tile.shape[0], point_offset,
                                             _stream()), "ts3_slice_accumulate")

    def finalize(self, w: LayerWeights):
        L.check(L.lib().ts3_slice_finalize(self.h, w.ref(), _stream()), "ts3_slice_finalize")

    def attention(self, w: LayerWeights):
        L.check(L.lib().ts3_token_attention(self.h, w.ref(), _stream()), "ts3_token_attention")

    def deslice(self, w: LayerWeights, x_chunk, out=None):
        self._check_x(x_chunk, "x_chunk")
        if out is None:
            out = torch.empty_like(x_chunk)
        self._check_x(out, "out")
        L.check(L.lib().ts3_deslice(self.h, w.ref(), _ptr(x_chunk), x_chunk.shape[0], _ptr(out), _stream()),
                "ts3_deslice")
        return out

    def forward(self, w: LayerWeights, x, tile: int, chunk: int | None = None, out=None):
        self._check_x(x)
        if out is None:
            out = torch.empty_like(x)
        self._check_x(out, "out")
        chunk = chunk or max(x.shape[0], 1)
        L.check(L.lib().ts3_layer_forward(self.h, w.ref(), _ptr(x), x.shape[0], tile, chunk, _ptr(out),
                                          _stream()), "ts3_layer_forward")
        return out

    def backward(self, w: LayerWeights, x, g, tile: int, dx=None):
        """Gradients of sum(g * x_out) after forward(w, x, ...) on this state:
        returns (dx, {dW2, db2, dW1, db1, dWq, dWk, dWv, dW3, db3}) as device
        float32 tensors shaped like x and the weights."""
        self._check_x(x)
        self._check_x(g, "g")
        if dx is None:
            dx = torch.empty_like(x)
        self._check_x(dx, "dx")
        grads = {}
        for n in L.GRAD_NAMES:
            wt = w.t[n[1:]]
            shape = wt.shape if wt is not None else {"db2": (self.H * self.M,), "db1": (self.H * self.dh,),
                                                     "db3": (self.C,)}[n]
            grads[n] = torch.empty(shape, device=x.device, dtype=torch.float32)
        gs = L.Grads(**{n: grads[n].data_ptr() for n in L.GRAD_NAMES})
        L.check(L.lib().ts3_layer_backward(self.h, w.ref(), _ptr(x), _ptr(g), x.shape[0], tile, _ptr(dx),
                                           ct.byref(gs), _stream()), "ts3_layer_backward")
        return dx, grads

    def get(self, which: int) -> np.ndarray:
        H, M, C, dh = self.H, self.M, self.C, self.dh
        shape = {L.TS3_S_RAW: (H, M, C), L.TS3_D: (H, M), L.TS3_S: (H, M, dh), L.TS3_S1: (H, M, dh),
                 L.TS3_ZP: (H, M, C), L.TS3_T_RAW: (H, M, dh)}[which]
        a = np.empty(shape, dtype=np.float32)
        L.check(L.lib().ts3_state_get(self.h, which, a.ctypes.data_as(ct.c_void_p), a.size, _stream()),
                "ts3_state_get")
        return a

    def get_spans(self, span0: int, nspan: int) -> np.ndarray:
        """Span partials [nspan, H, M, C+1] (columns :C sum w x, column C sum w),
        or [nspan, H, M, dh+1] (sum w x W1_h, then sum w) for a projected state."""
        a = np.empty((nspan, self.H, self.M, (self.dh if self.projected() else self.C) + 1), dtype=np.float32)
        L.check(L.lib().ts3_state_get_spans(self.h, span0, nspan, a.ctypes.data_as(ct.c_void_p), a.size,
                                            _stream()), "ts3_state_get_spans")
        return a

    def set_state(self, w: LayerWeights, Z: np.ndarray, b3: np.ndarray | None = None):
        Z = np.ascontiguousarray(Z, dtype=np.float32)
        b3p = None
        if b3 is not None:
            b3 = np.ascontiguousarray(b3, dtype=np.float32)
            b3p = b3.ctypes.data_as(ct.c_void_p)
        L.check(L.lib().ts3_state_set(self.h, w.ref(), L.TS3_ZP, Z.ctypes.data_as(ct.c_void_p), Z.size, b3p,
                                      _stream()), "ts3_state_set")


def layer_forward_noalloc(C, H, M, w: LayerWeights, x, tile: int, chunk: int, out, dh=None, temperature=0.5,
                          dtype="bf16", group_span=32768, eps=0.0, accum="fp32"):
    """ts3_layer_forward_noalloc: the whole layer over x into the preallocated
    out, with the library's fixed scratch array instead of a state object."""
    code, torch_dtype = _DTYPES[dtype]
    dh = C // H if dh is None else dh
    acc = {"fp32": L.TS3_ACCUM_FP32, "fp64": L.TS3_ACCUM_FP64}[accum]
    for t, name in ((x, "x"), (out, "out")):
        if not (t.is_cuda and t.dtype == torch_dtype and t.is_contiguous() and t.dim() == 2 and t.shape[1] == C):
            raise ValueError(f"{name} must be a contiguous cuda {torch_dtype} tensor [n, {C}]")
    desc = L.Desc(C=C, H=H, M=M, dh=dh, temperature=temperature, eps=eps, io_dtype=code, accum=acc,
                  group_span=group_span, max_points=x.shape[0])
    L.check(L.lib().ts3_layer_forward_noalloc(ct.byref(desc), w.ref(), _ptr(x), x.shape[0], tile, chunk, _ptr(out),
                                              _stream()), "ts3_layer_forward_noalloc")
    return out


def inv_tau_of(temperature: float) -> float:
    return 0.0 if math.isinf(temperature) else 1.0 / temperature
