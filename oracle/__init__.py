"""CPU float64 oracle for the Physics-Attention layer.

TEST INFRASTRUCTURE: imported only by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The GPU library never uses it.
"""
from .physics_attention import (build_state, deslice, layer_forward_fast, layer_forward_orig,
                                linear3_tokens, projected_accumulate, projected_finalize, slice_accumulate,
                                slice_finalize, slice_weights, token_attention, token_side)

__all__ = ["build_state", "deslice", "layer_forward_fast", "layer_forward_orig", "linear3_tokens",
           "projected_accumulate", "projected_finalize", "slice_accumulate", "slice_finalize", "slice_weights", "token_attention", "token_side"]
