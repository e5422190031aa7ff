"""Seeded layer weights: Xavier-uniform matrices, zero or small random biases.

Each matrix is one linear map with its own fan-in/fan-out:
  W2 [C, H*M]   slice-logit projection (Linear2)
  W1 [C, H*dh]  Linear1, applied to the slice tokens
  Wq, Wk, Wv [H, dh, dh]  per-head token-attention projections, no bias
  W3 [H*dh, C]  Linear3, applied to the slice tokens
Draw order is W2, W1, Wq, Wk, Wv, W3 from ``default_rng(seed)`` in float64,
stored as float32.  Biases b2 [H*M], b1 [H*dh], b3 [C] are zero unless
``bias_seed`` is given, in which case they are U(-0.1, 0.1).
"""
from __future__ import annotations

import numpy as np


def xavier_uniform(rng, shape, fan_in, fan_out):
    bound = np.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-bound, bound, size=shape)


def make_weights(C: int, H: int, M: int, dh: int, seed: int = 0, bias_seed: int | None = None):
    rng = np.random.default_rng(seed)
    HM, HD = H * M, H * dh
    w = {
        "W2": xavier_uniform(rng, (C, HM), C, HM),
        "W1": xavier_uniform(rng, (C, HD), C, HD),
        "Wq": xavier_uniform(rng, (H, dh, dh), dh, dh),
        "Wk": xavier_uniform(rng, (H, dh, dh), dh, dh),
        "Wv": xavier_uniform(rng, (H, dh, dh), dh, dh),
        "W3": xavier_uniform(rng, (HD, C), HD, C),
    }
    if bias_seed is None:
        w["b2"], w["b1"], w["b3"] = np.zeros(HM), np.zeros(HD), np.zeros(C)
    else:
        rb = np.random.default_rng(bias_seed)
        w["b2"] = rb.uniform(-0.1, 0.1, HM)
        w["b1"] = rb.uniform(-0.1, 0.1, HD)
        w["b3"] = rb.uniform(-0.1, 0.1, C)
    # stored as float32; the float64 views below hold exactly the stored values
    return {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in w.items()}


def make_block_weights(C: int, H: int, M: int, dh: int, F: int, seed: int = 0, bias_seed: int | None = None):
    """Weights of one pre-norm Transolver block: the Physics-Attention weights of
    ``make_weights(seed, bias_seed)`` plus LayerNorm affines ln1_g, ln1_b,
    ln2_g, ln2_b [C] and the feed-forward W_a [C, F], b_a [F], W_b [F, C],
    b_b [C].  W_a, W_b are Xavier-uniform from ``default_rng(seed + 7919)``;
    without ``bias_seed`` the gammas are one and the betas and biases zero,
    with it they are 1 + U(-0.1, 0.1) and U(-0.1, 0.1)."""
    w = make_weights(C, H, M, dh, seed, bias_seed)
    rng = np.random.default_rng(seed + 7919)
    w["Wa"] = xavier_uniform(rng, (C, F), C, F)
    w["Wb"] = xavier_uniform(rng, (F, C), F, C)
    if bias_seed is None:
        w["ln1_g"], w["ln2_g"] = np.ones(C), np.ones(C)
        w["ln1_b"], w["ln2_b"], w["ba"], w["bb"] = np.zeros(C), np.zeros(C), np.zeros(F), np.zeros(C)
    else:
        rb = np.random.default_rng(bias_seed + 7919)
        w["ln1_g"], w["ln1_b"] = 1.0 + rb.uniform(-0.1, 0.1, C), rb.uniform(-0.1, 0.1, C)
        w["ln2_g"], w["ln2_b"] = 1.0 + rb.uniform(-0.1, 0.1, C), rb.uniform(-0.1, 0.1, C)
        w["ba"], w["bb"] = rb.uniform(-0.1, 0.1, F), rb.uniform(-0.1, 0.1, C)
    return {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in w.items()}
