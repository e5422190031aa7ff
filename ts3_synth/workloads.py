"""Named synthetic workloads (sizes follow the paper's meshes and model shape).

Each workload fixes the geometry, the feature width C, heads H, slices per head
M, head dim dh, temperature tau, storage dtype and the tile/chunk sizes the
layer runs with.  ``features(name, start, n)`` returns rows ``[start, start+n)``
of the input x in float64 after storage rounding (the exact values the GPU
sees), generated chunk by chunk so any window can be rebuilt independently.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import geometry as G
from .features import feature_map, point_features, round_bf16, to_f32


@dataclass(frozen=True)
class Workload:
    name: str
    geometry: str          # "ellipsoid" | "car_surface" | "volume"
    seed: int
    N: int
    C: int
    H: int
    M: int
    dh: int
    tau: float
    dtype: str             # "fp32" | "bf16"
    tile: int
    chunk: int
    group_span: int
    source_N: int = 0      # > 0: the N points are a seeded draw from a mesh of this many
    subset_seed: int = 0   # seed of that draw (numpy default_rng)


WORKLOADS = {
    # one Physics-Attention layer, fp32, ellipsoid surface, one tile
    "ellipsoid_4k_fp32": Workload("ellipsoid_4k_fp32", "ellipsoid", 2, 4096, 64, 4, 16, 16, 0.5,
                                  "fp32", 4096, 4096, 4096),
    # one layer, bf16 storage, 1M surface points in 65,536-point tiles
    "ellipsoid_1m_bf16": Workload("ellipsoid_1m_bf16", "ellipsoid", 2, 1_000_000, 128, 8, 32, 16, 0.5,
                                  "bf16", 65_536, 65_536, 16_384),
    # one layer of an 8-block stack on a 10M-point car surface (per-layer shape)
    "car_10m_bf16": Workload("car_10m_bf16", "car_surface", 3, 10_000_000, 256, 8, 64, 32, 0.5,
                             "bf16", 1_000_000, 1_000_000, 31_250),
    # a training step of one layer (forward and backward, float32) on 2M volume
    # points drawn uniformly without replacement from a 160M-point volume mesh
    # (the geometry-amortized training of section 3.2 samples subsets of the
    # full mesh)
    "volume_2m_fp32": Workload("volume_2m_fp32", "volume", 5, 2_000_000, 128, 8, 64, 16, 0.5,
                               "fp32", 1_000_000, 1_000_000, 15_625, source_N=160_000_000, subset_seed=6),
    # cached-state inference over 100M volume points, 1M-point tiles and chunks
    "volume_100m_bf16": Workload("volume_100m_bf16", "volume", 4, 100_000_000, 128, 8, 64, 16, 0.5,
                                 "bf16", 1_000_000, 1_000_000, 15_625),
}


def _points(w: Workload, k: int, n: int, body=None):
    if w.geometry == "ellipsoid":
        return G.ellipsoid_surface_chunk(w.seed, k, n)
    if w.geometry == "car_surface":
        return G.car_surface_chunk(w.seed, k, n, body)
    if w.geometry == "volume":
        return G.volume_chunk(w.seed, k, n, body)
    raise ValueError(w.geometry)


def bbox(w: Workload, body=None):
    if w.geometry == "ellipsoid":
        return G.ellipsoid_bbox()
    if w.geometry == "car_surface":
        return (body or G.CarBody()).bbox()
    return G.volume_bbox()


def round_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16(x) if dtype == "bf16" else to_f32(x).astype(np.float64)


def features_chunk(w: Workload, k: int, n: int | None = None, body=None, R=None) -> np.ndarray:
    """Stored-precision features (float64 values) of the first ``n`` points of chunk k."""
    n = G.CHUNK if n is None else n
    body = body if body is not None or w.geometry == "ellipsoid" else G.CarBody()
    lo, hi = bbox(w, body)
    p = _points(w, k, n, body)
    return round_storage(point_features(p, lo, hi, w.C, R), w.dtype)


def features(w: Workload, start: int, n: int) -> np.ndarray:
    """Rows [start, start+n) of x (float64 values after storage rounding)."""
    body = None if w.geometry == "ellipsoid" else G.CarBody()
    R = feature_map(w.C)
    out = np.empty((n, w.C))
    pos = start
    while pos < start + n:
        k, off = divmod(pos, G.CHUNK)
        take = min(G.CHUNK - off, start + n - pos)
        # samplers are prefix-stable, so generating off+take points is enough
        full = features_chunk(w, k, off + take, body, R)
        out[pos - start:pos - start + take] = full[off:off + take]
        pos += take
    return out


def subset_indices(w: Workload) -> np.ndarray:
    """Mesh rows of a drawn workload: w.N indices drawn uniformly without
    replacement from range(w.source_N) by numpy's default_rng(w.subset_seed),
    sorted ascending (so the subset keeps the mesh's order)."""
    if not w.source_N:
        return np.arange(w.N, dtype=np.int64)
    return np.sort(np.random.default_rng(w.subset_seed).choice(w.source_N, w.N, replace=False)).astype(np.int64)


def small_features(w: Workload, n: int) -> np.ndarray:
    """First n rows of x (the samplers are prefix-stable, so this is features(w, 0, n))."""
    return features(w, 0, n)
