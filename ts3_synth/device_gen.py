"""Device-side generator for meshes too large to build on the host.

Same recipe as ``geometry`` + ``features`` (volume points uniform in the box
minus the car-like body, Fourier features, fixed Gaussian map, LayerNorm,
float64 arithmetic, round-to-nearest-even storage), drawn with torch's
counter-based generator on the device instead of numpy's.  Chunk k of a mesh
uses ``torch.Generator(device).manual_seed(seed * 2**32 + k)``, so chunks are
independent and any chunk can be regenerated alone.  The body shape and the
feature map are the numpy ones, bit for bit.
"""
from __future__ import annotations

import numpy as np
import torch

from . import geometry as G
from .features import LN_EPS, N_FREQ, feature_map

ROUND = 1 << 20


class DeviceVolume:
    def __init__(self, seed: int, C: int, device="cuda", dtype=torch.bfloat16):
        self.seed, self.C, self.device, self.dtype = seed, C, torch.device(device), dtype
        body = G.CarBody()
        f64 = dict(device=self.device, dtype=torch.float64)
        self.v = torch.tensor(body.v, **f64)
        self.alpha = torch.tensor(body.alpha, **f64)
        self.inv2s2 = torch.tensor(1.0 / (2.0 * body.sigma ** 2), **f64)
        self.centre = torch.tensor(G.BODY_CENTRE, **f64)
        self.axes = torch.tensor(G.BODY_AXES, **f64)
        self.lo = torch.tensor(G.VOLUME_BOX_LO, **f64)
        self.hi = torch.tensor(G.VOLUME_BOX_HI, **f64)
        self.R = torch.tensor(feature_map(C), **f64)
        self.freq = torch.tensor(np.pi * 2.0 ** (np.arange(N_FREQ) / 3.0), **f64)

    def _radius(self, u):
        e = G.BODY_EXPONENT
        rse = ((u / self.axes).abs() ** e).sum(dim=1) ** (-1.0 / e)
        d2 = (2.0 - 2.0 * (u @ self.v.T)).clamp_min(0.0)
        return rse * (1.0 + torch.exp(-d2 * self.inv2s2) @ self.alpha)

    def points(self, k: int, n: int = G.CHUNK):
        gen = torch.Generator(device=self.device)
        gen.manual_seed(self.seed * (1 << 32) + k)
        parts, got = [], 0
        while got < n:
            p = self.lo + torch.rand((ROUND, 3), generator=gen, device=self.device,
                                     dtype=torch.float64) * (self.hi - self.lo)
            r = p - self.centre
            dist = r.norm(dim=1)
            u = r / dist.clamp_min(1e-300)[:, None]
            q = p[dist >= self._radius(u)]
            parts.append(q[:n - got])
            got += len(parts[-1])
        return torch.cat(parts)

    def features(self, p):
        q = 2.0 * (p - self.lo) / (self.hi - self.lo) - 1.0
        arg = q[:, :, None] * self.freq
        phi = torch.cat([torch.sin(arg), torch.cos(arg)], dim=2).reshape(len(p), 6 * N_FREQ)
        z = phi @ self.R
        mu = z.mean(dim=1, keepdim=True)
        var = ((z - mu) ** 2).mean(dim=1, keepdim=True)
        return ((z - mu) / torch.sqrt(var + LN_EPS)).to(torch.float32).to(self.dtype)

    def fill(self, x: torch.Tensor, progress=None):
        """Write chunks 0.. of the mesh into the preallocated device tensor x [N, C]."""
        N = x.shape[0]
        for k in range((N + G.CHUNK - 1) // G.CHUNK):
            n = min(G.CHUNK, N - k * G.CHUNK)
            x[k * G.CHUNK:k * G.CHUNK + n] = self.features(self.points(k, n))
            if progress and (k % 10 == 9 or k * G.CHUNK + n == N):
                progress(k + 1)
        return x


    def gather(self, x: torch.Tensor, indices, source_N: int, progress=None):
        """Write rows ``indices`` (sorted, distinct, < source_N) of a source_N-point
        mesh into x [len(indices), C]: every chunk holding a drawn row is
        generated with the same calls ``fill`` makes for that mesh and the drawn
        rows are selected from it, so they are the rows ``fill`` writes at those
        positions."""
        idx = np.asarray(indices, dtype=np.int64)
        if len(idx) != x.shape[0]:
            raise ValueError("x must have one row per index")
        if len(idx) and ((np.diff(idx) <= 0).any() or idx[0] < 0 or idx[-1] >= source_N):
            raise ValueError("indices must be sorted, distinct and in [0, source_N)")
        chunks = idx // G.CHUNK
        bounds = np.searchsorted(chunks, np.arange(chunks[-1] + 2)) if len(idx) else np.zeros(1, np.int64)
        for k in range(len(bounds) - 1):
            a, b = int(bounds[k]), int(bounds[k + 1])
            if a == b:
                continue
            local = torch.from_numpy(idx[a:b] - k * G.CHUNK).to(self.device)
            n = min(G.CHUNK, source_N - k * G.CHUNK)
            x[a:b] = self.features(self.points(k, n))[local]
            if progress and (k % 20 == 19 or b == len(idx)):
                progress(k + 1)
        return x


class DeviceSurface(DeviceVolume):
    """Points on the car-like body's surface (uniform in direction, the host
    recipe of ``geometry.car_surface_chunk``), features over the body's padded
    bounding box; chunk k uses ``manual_seed(seed * 2**32 + k)``."""

    def __init__(self, seed: int, C: int, device="cuda", dtype=torch.bfloat16):
        super().__init__(seed, C, device, dtype)
        lo, hi = G.CarBody().bbox()
        self.lo = torch.tensor(lo, device=self.device, dtype=torch.float64)
        self.hi = torch.tensor(hi, device=self.device, dtype=torch.float64)

    def points(self, k: int, n: int = G.CHUNK):
        gen = torch.Generator(device=self.device)
        gen.manual_seed(self.seed * (1 << 32) + k)
        g = torch.randn((n, 3), generator=gen, device=self.device, dtype=torch.float64)
        u = g / g.norm(dim=1, keepdim=True)
        return self.centre + self._radius(u)[:, None] * u
