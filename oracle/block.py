"""Plain float64 CPU oracle for a stack of Transolver blocks.

TEST INFRASTRUCTURE.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU baseline may import this module.  It shares no code with the
GPU path and the GPU path never calls it.

Transolver-3 stacks L blocks of Physics-Attention and a feed-forward network
(the model context of section 3 and the 8-layer configuration of Table 7).
The paper does not spell out where the normalisations and residuals go; this
oracle takes the pre-norm residual form of the Transolver family:

  y   = x + PA(LN1(x))                       (PA: ``layer_forward_fast``)
  out = y + W_b^T GELU(W_a^T LN2(y) + b_a) + b_b

with LayerNorm over the C channels (affine gamma, beta; eps = 1e-5), GELU in
its exact form x * Phi(x) = x/2 (1 + erf(x / sqrt 2)), and a 4C-wide hidden
layer.  Shapes: gamma, beta [C]; W_a [C, F], b_a [F]; W_b [F, C], b_b [C].

Pinned in ``tests/test_oracle_block.py``: LayerNorm against torch's float64
layer_norm and its zero-mean / unit-variance property, GELU against the
normal CDF of scipy and its odd-part identity, the MLP against loops, and the
block's residual structure (zero output weights give the identity; a block of
a block equals two stacked blocks).
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

from .physics_attention import build_state, deslice, layer_forward_fast

LN_EPS = 1e-5


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def layer_norm(x, gamma, beta, eps: float = LN_EPS):
    """(x - mean) / sqrt(var + eps) * gamma + beta over the last axis (biased var)."""
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * _f64(gamma) + _f64(beta)


def gelu(x):
    """Exact GELU: x * Phi(x) with Phi the standard normal CDF."""
    x = _f64(x)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def mlp(x, Wa, ba, Wb, bb):
    """W_b^T GELU(W_a^T x + b_a) + b_b for rows x [N, C]."""
    return gelu(_f64(x) @ _f64(Wa) + _f64(ba)) @ _f64(Wb) + _f64(bb)


def block_forward(x, B, H: int, M: int, inv_tau: float, tile: int | None = None):
    """One pre-norm Transolver block over the whole mesh x [N, C].  B holds the
    Physics-Attention weights (``physics_attention`` names) and ln1_g, ln1_b,
    ln2_g, ln2_b, Wa, ba, Wb, bb."""
    x = _f64(x)
    y = x + layer_forward_fast(layer_norm(x, B["ln1_g"], B["ln1_b"]), B, H, M, inv_tau, tile=tile)
    return y + mlp(layer_norm(y, B["ln2_g"], B["ln2_b"]), B["Wa"], B["ba"], B["Wb"], B["bb"])


def stack_forward(x, blocks, H: int, M: int, inv_tau: float, tile: int | None = None):
    """The blocks in order; returns the last block's output."""
    for B in blocks:
        x = block_forward(x, B, H, M, inv_tau, tile)
    return x


def stack_states(x, blocks, H: int, M: int, inv_tau: float):
    """Each block's cached physical state Z [H, M, C] from a forward over the
    mesh x (section 3.3, physical state caching)."""
    Zs = []
    x = _f64(x)
    for B in blocks:
        xn = layer_norm(x, B["ln1_g"], B["ln1_b"])
        Z = build_state(xn, B, H, M, inv_tau, tile=len(x))["Z"]
        Zs.append(Z)
        y = x + deslice(xn, B["W2"], B["b2"], Z, B["b3"], H, M, inv_tau)
        x = y + mlp(layer_norm(y, B["ln2_g"], B["ln2_b"]), B["Wa"], B["ba"], B["Wb"], B["bb"])
    return Zs


def stack_decode(q, blocks, Zs, H: int, M: int, inv_tau: float):
    """Outputs at query points q [n, C] from cached states: every block
    decodes its Physics-Attention from Z (Eq. (5)) instead of re-slicing the
    mesh.  Query points may be any points; with the mesh's own points this is
    the stack's forward."""
    x = _f64(q)
    for B, Z in zip(blocks, Zs):
        y = x + deslice(layer_norm(x, B["ln1_g"], B["ln1_b"]), B["W2"], B["b2"], Z, B["b3"], H, M, inv_tau)
        x = y + mlp(layer_norm(y, B["ln2_g"], B["ln2_b"]), B["Wa"], B["ba"], B["Wb"], B["bb"])
    return x
