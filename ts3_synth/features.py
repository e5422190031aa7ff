"""Point features fed to the layer, and host-side storage rounding.

Recipe: coordinates are min-max scaled to [-1, 1]^3 over the geometry's fixed
bounding box (the coordinate scaling of Appendix A.2), expanded to 16
frequencies of sin/cos per axis (96 features), mapped to C channels by a fixed
seeded Gaussian matrix, and normalised per point by a LayerNorm without affine
parameters.  All float64; storage rounding is round-to-nearest-even.
"""
from __future__ import annotations

import numpy as np

N_FREQ = 16
FEATURE_MAP_SEED = 1
LN_EPS = 1e-5


def fourier_features(p: np.ndarray, lo: np.ndarray, hi: np.ndarray) -> np.ndarray:
    q = 2.0 * (p - lo) / (hi - lo) - 1.0
    f = np.pi * 2.0 ** (np.arange(N_FREQ) / 3.0)
    arg = q[:, :, None] * f[None, None, :]          # [n, 3, 16]
    phi = np.concatenate([np.sin(arg), np.cos(arg)], axis=2)  # [n, 3, 32]
    return phi.reshape(len(p), 6 * N_FREQ)


def feature_map(C: int) -> np.ndarray:
    rng = np.random.default_rng(FEATURE_MAP_SEED)
    return rng.standard_normal((6 * N_FREQ, C)) / np.sqrt(6 * N_FREQ)


def layer_norm(z: np.ndarray, eps: float = LN_EPS) -> np.ndarray:
    mu = z.mean(axis=1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=1, keepdims=True)
    return (z - mu) / np.sqrt(var + eps)


def point_features(p: np.ndarray, lo, hi, C: int, R: np.ndarray | None = None) -> np.ndarray:
    R = feature_map(C) if R is None else R
    return layer_norm(fourier_features(p, lo, hi) @ R)


# ----------------------------------------------------------------- rounding

def to_f32(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((u.astype(np.uint64) + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(np.asarray(a, dtype=np.float32))
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """float64 -> float32 -> bfloat16 -> float64 values (the stored input)."""
    return bf16_bits_to_f32(f32_to_bf16_bits(to_f32(a))).astype(np.float64)
