"""Seeded synthetic mesh points.

The paper evaluates on aerodynamic meshes (a wing-body surface of ~0.4M
points, car surfaces of ~1-9M points and car volume meshes of ~20-160M cells,
section 4 "Benchmarks" and Appendix A.1).  None of those datasets is used here;
these generators produce points with the same sizes and the same kinds of
geometry (a smooth closed surface, a bumpy car-like body, and the air volume
around that body) so the layer sees inputs of the paper's shape.

Every generator is chunked: chunk ``k`` holds points ``[k*CHUNK, (k+1)*CHUNK)``
and is drawn from ``np.random.default_rng([seed, k])``, so any chunk can be
regenerated on its own and the points do not depend on how the layer later
tiles them.  All arithmetic is float64.
"""
from __future__ import annotations

import numpy as np

CHUNK = 1_000_000
# Rejection samplers draw candidates in rounds of this fixed size, so the first
# n accepted points of a chunk do not depend on how many points were requested.
ROUND = 1 << 16

ELLIPSOID_AXES = (2.0, 0.8, 0.6)

# Car-like body: a superellipsoid of length 4.5 m with Gaussian bumps.
BODY_CENTRE = np.array([0.0, 0.0, 0.9])
BODY_AXES = np.array([2.25, 0.9, 0.7])
BODY_EXPONENT = 4.0
BODY_BUMPS = 200
BODY_BUMP_SEED = 3

# Air volume around the body: a 10 x 4 x 3 m box.
VOLUME_BOX_LO = np.array([-3.5, -2.0, 0.0])
VOLUME_BOX_HI = np.array([6.5, 2.0, 3.0])


def _unit_vectors(rng: np.random.Generator, n: int) -> np.ndarray:
    g = rng.standard_normal((n, 3))
    return g / np.linalg.norm(g, axis=1, keepdims=True)


def ellipsoid_bbox(axes=ELLIPSOID_AXES):
    a = np.asarray(axes, dtype=np.float64)
    return -a, a


def ellipsoid_surface_chunk(seed: int, k: int, n: int, axes=ELLIPSOID_AXES) -> np.ndarray:
    """``n`` points of chunk ``k``, area-uniform on the ellipsoid surface.

    A direction u uniform on the sphere maps to p = (a u_x, b u_y, c u_z); the
    area element of that map is proportional to
    sqrt((bc u_x)^2 + (ac u_y)^2 + (ab u_z)^2), which is at most a*b for
    a >= b >= c, so accepting with that ratio gives area-uniform points.
    """
    a, b, c = axes
    rng = np.random.default_rng([seed, k])
    out = np.empty((n, 3))
    got = 0
    while got < n:
        m = ROUND
        u = _unit_vectors(rng, m)
        dens = np.sqrt((b * c * u[:, 0]) ** 2 + (a * c * u[:, 1]) ** 2 + (a * b * u[:, 2]) ** 2)
        keep = rng.random(m) * (a * b) < dens
        p = u[keep] * np.array([a, b, c])
        take = min(n - got, len(p))
        out[got:got + take] = p[:take]
        got += take
    return out


class CarBody:
    """Star-shaped car-like body: superellipsoid radius times a bump field."""

    def __init__(self, seed: int = BODY_BUMP_SEED, n_bumps: int = BODY_BUMPS):
        rng = np.random.default_rng(seed)
        self.v = _unit_vectors(rng, n_bumps)
        self.alpha = rng.uniform(-0.04, 0.04, n_bumps)
        self.sigma = rng.uniform(0.05, 0.25, n_bumps)

    def radius(self, u: np.ndarray) -> np.ndarray:
        """Surface radius along unit directions ``u`` [n, 3]."""
        e = BODY_EXPONENT
        rse = (np.abs(u[:, 0] / BODY_AXES[0]) ** e + np.abs(u[:, 1] / BODY_AXES[1]) ** e
               + np.abs(u[:, 2] / BODY_AXES[2]) ** e) ** (-1.0 / e)
        bump = np.empty(len(u))
        step = 65536
        for s in range(0, len(u), step):
            uu = u[s:s + step]
            d2 = np.maximum(2.0 - 2.0 * (uu @ self.v.T), 0.0)  # |u - v_k|^2 on the sphere
            bump[s:s + step] = np.exp(-d2 / (2.0 * self.sigma ** 2)) @ self.alpha
        return rse * (1.0 + bump)

    def bbox(self):
        # The bumps change the radius by at most sum|alpha| relative; use a padded box.
        pad = 1.0 + np.abs(self.alpha).sum()
        return BODY_CENTRE - BODY_AXES * pad, BODY_CENTRE + BODY_AXES * pad


def car_surface_chunk(seed: int, k: int, n: int, body: CarBody | None = None) -> np.ndarray:
    """``n`` points of chunk ``k`` on the car-like surface (uniform in direction,
    not area-uniform)."""
    body = body or CarBody()
    rng = np.random.default_rng([seed, k])
    u = _unit_vectors(rng, n)
    return BODY_CENTRE + body.radius(u)[:, None] * u


def volume_chunk(seed: int, k: int, n: int, body: CarBody | None = None) -> np.ndarray:
    """``n`` points of chunk ``k``, uniform in the box minus the car-like body."""
    body = body or CarBody()
    rng = np.random.default_rng([seed, k])
    out = np.empty((n, 3))
    got = 0
    while got < n:
        m = ROUND
        p = VOLUME_BOX_LO + rng.random((m, 3)) * (VOLUME_BOX_HI - VOLUME_BOX_LO)
        r = p - BODY_CENTRE
        dist = np.linalg.norm(r, axis=1)
        u = r / np.maximum(dist, 1e-300)[:, None]
        keep = dist >= body.radius(u)
        q = p[keep]
        take = min(n - got, len(q))
        out[got:got + take] = q[:take]
        got += take
    return out


def volume_bbox():
    return VOLUME_BOX_LO.copy(), VOLUME_BOX_HI.copy()
