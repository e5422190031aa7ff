"""Process-pool driver of the float64 oracle, for samples of a million points.

TEST INFRASTRUCTURE (see ``physics_attention.py``): only the tests, the smoke
check and the benchmark's CPU baseline use it.  It adds no arithmetic of its
own.  Workers run the oracle's ``slice_accumulate`` (or
``projected_accumulate``) on one tile, or its ``deslice`` on one chunk.  The
parent adds the tile terms in tile-index order (Eq. (4): the state's sums
are additive over parts of the mesh), in the same
order and from the same zero start as ``build_state``, so both give bitwise
equal results.  It then runs the token side (``token_side``) once.

Workers are started with "spawn" (they never inherit a GPU context) and each
limits its BLAS to one thread, so a pool of P workers uses P cores.
"""
from __future__ import annotations

import multiprocessing as mp
import os
from concurrent.futures import ProcessPoolExecutor

import numpy as np

from . import physics_attention as PA


def _init():
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _tile_sum(args):
    x, W2, b2, H, M, inv_tau = args
    return PA.slice_accumulate(np.asarray(x, dtype=np.float64), W2, b2, H, M, inv_tau)


def _tile_psum(args):
    x, W2, b2, W1, H, M, inv_tau = args
    return PA.projected_accumulate(np.asarray(x, dtype=np.float64), W2, b2, W1, H, M, inv_tau)


def _tile_decode(args):
    x, W2, b2, Z, b3, H, M, inv_tau = args
    return PA.deslice(np.asarray(x, dtype=np.float64), W2, b2, Z, b3, H, M, inv_tau)


def host_cores() -> int:
    """Cores this process may run on (the affinity mask, not the machine's count)."""
    return len(os.sched_getaffinity(0))


class OraclePool:
    """``with OraclePool(P) as pool: st = pool.state(x, W, ...)``.

    Inputs are passed to workers as float32 when that is exact (bf16- and
    fp32-stored features are), halving what is pickled; workers compute in
    float64 as the oracle does.
    """

    def __init__(self, workers: int | None = None):
        self.workers = max(1, workers or min(host_cores(), 16))
        self.ex = ProcessPoolExecutor(self.workers, mp_context=mp.get_context("spawn"), initializer=_init)

    def close(self):
        self.ex.shutdown(wait=True, cancel_futures=True)

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    @staticmethod
    def _pack(x):
        x = np.asarray(x)
        if x.dtype == np.float64:
            x32 = x.astype(np.float32)
            if np.array_equal(x32, x):
                return x32
        return x

    def tile_sums(self, x, W2, b2, H: int, M: int, inv_tau: float, tile: int):
        """[(s_raw_t, d_t)] for the tiles [t0, t0 + tile) of x, in tile order."""
        jobs = [(self._pack(x[t0:t0 + tile]), W2, b2, H, M, inv_tau) for t0 in range(0, len(x), tile)]
        return list(self.ex.map(_tile_sum, jobs))

    def sums(self, parts, W2, b2, H: int, M: int, inv_tau: float):
        """[(s_raw, d)] of ``slice_accumulate`` over each point set in ``parts``."""
        return list(self.ex.map(_tile_sum, [(self._pack(p), W2, b2, H, M, inv_tau) for p in parts]))

    def projected_sums(self, parts, W2, b2, W1, H: int, M: int, inv_tau: float):
        """[(t_raw, d)] of ``projected_accumulate`` over each point set in ``parts``."""
        return list(self.ex.map(_tile_psum, [(self._pack(p), W2, b2, W1, H, M, inv_tau) for p in parts]))

    def projected_tile_sums(self, x, W2, b2, W1, H: int, M: int, inv_tau: float, tile: int):
        """[(t_raw_t, d_t)] for the tiles [t0, t0 + tile) of x, in tile order."""
        return self.projected_sums([x[t0:t0 + tile] for t0 in range(0, len(x), tile)], W2, b2, W1, H, M, inv_tau)

    def state(self, x, W, H: int, M: int, inv_tau: float, tile: int = 65536, eps: float = 0.0):
        """The oracle's ``build_state(x, W, H, M, inv_tau, tile, eps)``, tiles in parallel."""
        C = np.asarray(x).shape[1]
        parts = self.tile_sums(x, W["W2"], W["b2"], H, M, inv_tau, tile) if len(x) > tile else \
            [PA.slice_accumulate(np.asarray(x, dtype=np.float64), W["W2"], W["b2"], H, M, inv_tau)]
        s_raw = sum((t[0] for t in parts), np.zeros((H, M, C)))
        d = sum((t[1] for t in parts), np.zeros((H, M)))
        return {"s_raw": s_raw, "d": d, **PA.token_side(s_raw, d, W, H, eps)}

    def decode(self, x, W2, b2, Z, b3, H: int, M: int, inv_tau: float, chunk: int = 65536):
        """The oracle's ``deslice`` over x, chunks in parallel -> [N, C]."""
        jobs = [(self._pack(x[c0:c0 + chunk]), W2, b2, Z, b3, H, M, inv_tau) for c0 in range(0, len(x), chunk)]
        parts = list(self.ex.map(_tile_decode, jobs))
        return np.concatenate(parts) if parts else np.zeros((0, np.asarray(Z).shape[2]))
