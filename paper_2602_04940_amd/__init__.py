"""Transolver-3 Physics-Attention layer on MI355X (gfx950).

The layer runs in ``libts3.so`` (HIP kernels behind the C ABI of
``include/ts3.h``); ``layer.PhysicsAttention`` marshals torch tensors into it.
Importing this package loads nothing; the library is loaded on first use.
"""
__all__ = ["PhysicsAttention", "LayerWeights", "TransolverStack", "BlockWeights"]


def __getattr__(name):
    if name in ("PhysicsAttention", "LayerWeights"):
        from . import layer
        return getattr(layer, name)
    if name in ("TransolverStack", "BlockWeights"):
        from . import stack
        return getattr(stack, name)
    raise AttributeError(name)
