"""Python face of the Transolver block stack in libts3 (include/ts3.h,
ts3_stack_*): argument marshalling only; every step runs in the library."""
from __future__ import annotations

import ctypes as ct

import torch

from . import _lib as L
from .layer import LayerWeights, PhysicsAttention, _ptr, _stream


class BlockWeights:
    """Device float32 copies of one block's weights: the Physics-Attention
    weights plus ln1_g, ln1_b, ln2_g, ln2_b, Wa, ba, Wb, bb."""

    def __init__(self, weights: dict, device="cuda"):
        self.pa = LayerWeights(weights, device)
        self.t = {n: torch.as_tensor(weights[n]).to(device=device, dtype=torch.float32).contiguous()
                  for n in L.BLOCK_EXTRA_NAMES}
        self.struct = L.BlockWeights(pa=self.pa.struct, **{n: self.t[n].data_ptr() for n in L.BLOCK_EXTRA_NAMES})


class TransolverStack:
    """n_blocks pre-norm blocks of Physics-Attention + feed-forward (bf16)."""

    def __init__(self, C, H, M, n_blocks, hidden=None, dh=None, temperature=0.5, group_span=32768,
                 max_points=1 << 20, accum="fp32"):
        self.C, self.H, self.M, self.L = C, H, M, n_blocks
        self.F = hidden or 4 * C
        self.dh = dh or C // H
        acc = {"fp32": L.TS3_ACCUM_FP32, "fp64": L.TS3_ACCUM_FP64}[accum]
        self.desc = L.Desc(C=C, H=H, M=M, dh=self.dh, temperature=temperature, eps=0.0, io_dtype=L.TS3_BF16,
                           accum=acc, group_span=group_span, max_points=max_points)
        h = ct.c_void_p()
        L.check(L.lib().ts3_stack_create(ct.byref(self.desc), n_blocks, self.F, ct.byref(h)), "ts3_stack_create")
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            L.check(L.lib().ts3_stack_free(self.h), "ts3_stack_free")
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

    def _blocks(self, blocks):
        if len(blocks) != self.L:
            raise ValueError(f"{self.L} blocks expected")
        arr = (L.BlockWeights * self.L)(*[b.struct for b in blocks])
        return arr

    def _check(self, x):
        if not (x.is_cuda and x.dtype == torch.bfloat16 and x.is_contiguous() and x.dim() == 2
                and x.shape[1] == self.C):
            raise ValueError(f"x must be a contiguous cuda bfloat16 tensor [n, {self.C}]")

    def bytes(self) -> int:
        b = ct.c_int64()
        L.check(L.lib().ts3_stack_bytes(self.h, ct.byref(b)), "ts3_stack_bytes")
        return b.value

    def forward(self, blocks, x, tile: int, chunk: int):
        """x (bf16 [N, C]) is overwritten with the stack's output."""
        self._check(x)
        arr = self._blocks(blocks)
        L.check(L.lib().ts3_stack_forward(self.h, arr, _ptr(x), x.shape[0], tile, chunk, _stream()),
                "ts3_stack_forward")
        return x

    def decode(self, blocks, q, chunk: int):
        """Query points q (bf16 [n, C]) through every block from the cached states (in place)."""
        self._check(q)
        arr = self._blocks(blocks)
        L.check(L.lib().ts3_stack_decode(self.h, arr, _ptr(q), q.shape[0], chunk, _stream()), "ts3_stack_decode")
        return q

    def feedforward(self, blocks, l: int, x, pa, xn_next=None):
        """Block l's feed-forward half in place on x given its attention output pa."""
        self._check(x)
        self._check(pa)
        if xn_next is not None:
            self._check(xn_next)
        arr = self._blocks(blocks)
        L.check(L.lib().ts3_stack_feedforward(self.h, arr, l, _ptr(x), _ptr(pa), x.shape[0], _ptr(xn_next),
                                              _stream()), "ts3_stack_feedforward")
        return x

    def layer(self, l: int) -> PhysicsAttention:
        """Block l's layer state as a (non-owning) PhysicsAttention view."""
        h = ct.c_void_p()
        L.check(L.lib().ts3_stack_layer(self.h, l, ct.byref(h)), "ts3_stack_layer")
        view = PhysicsAttention.__new__(PhysicsAttention)
        view.C, view.H, view.M, view.dh = self.C, self.H, self.M, self.dh
        view.dtype_name, view.torch_dtype = "bf16", torch.bfloat16
        view.h = h
        view.close = lambda: None
        return view
