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
