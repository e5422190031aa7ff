"""Plain float64 CPU oracle for the backward of one Physics-Attention layer.

TEST INFRASTRUCTURE.  Only the tests may import this module.  It shares no
code with the GPU path and the GPU path never calls it.

The paper trains with every tile's slice computation checkpointed (section
3.2, "Geometry slice tiling", and the Checkpoint steps of Algorithm 1): the
slice weights are never stored and are recomputed tile by tile when the
gradients are formed.  This oracle takes the chain rule through the fast
(slice, then project) form of the forward in that shape.  Given the output
gradient g = dL/dx_out [N, C]:

  pass B1 (over tiles)  dZ[h, m] = sum_i w[i, h, m] g_i            (deslice)
                        db3      = sum_i g_i
  token side            Z = s' W3_h  ->  ds', dW3
                        s' = Attention(s)  ->  ds, dWq, dWk, dWv
                        s = mean W1_h + b1_h  ->  dmean, dW1, db1
                        mean = s_raw / d  ->  ds_raw = dmean / d,
                                              dd = -sum_c dmean * mean / d
  pass B2 (over tiles)  dw[i, h, m] = g_i . Z[h, m] + x_i . ds_raw[h, m] + dd[h, m]
                        dz = inv_tau * w * (dw - sum_m w dw)       (softmax)
                        dx_i = dz_i W2^T + sum_{h,m} w[i, h, m] ds_raw[h, m]
                        dW2 = sum_i x_i^T dz_i,  db2 = sum_i dz_i

Notation and weight layout as in ``physics_attention``.  Pinned in
``tests/test_oracle_backward.py`` by central finite differences of the float64
forward on small problems, tile independence, and invariants that hold for any
input (the logit gradients of a head sum to zero over its slices; the bias b3
receives the column sum of g).
"""
from __future__ import annotations

import numpy as np

from .physics_attention import build_state, slice_weights


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def _mean_and_den(s_raw, d, eps):
    den = (d + eps)[:, :, None]
    mean = np.divide(s_raw, den, out=np.zeros_like(s_raw), where=den > 0)
    return mean, den


def dZ_accumulate(x_tile, g_tile, W2, b2, H: int, M: int, inv_tau: float):
    """Pass B1 on one tile: sum_i w_i^T g_i -> [H, M, C] (w recomputed)."""
    w = slice_weights(x_tile, W2, b2, H, M, inv_tau)
    return np.einsum("nhm,nc->hmc", w, _f64(g_tile))


def token_backward(state, dZ, W, H: int, eps: float = 0.0):
    """Gradients through Linear3, the per-head attention, Linear1 and the
    normalisation d^-1 s_raw, for the cached state of ``build_state``.

    Returns ds_raw [H, M, C], dd [H, M] and the token-side weight gradients.
    """
    dZ = _f64(dZ)
    s_raw, d, s, s1 = (_f64(state[k]) for k in ("s_raw", "d", "s", "s1"))
    C = s_raw.shape[2]
    dh = C // H
    W1, W3 = _f64(W["W1"]), _f64(W["W3"])
    Wq, Wk, Wv = _f64(W["Wq"]), _f64(W["Wk"]), _f64(W["Wv"])
    mean, den = _mean_and_den(s_raw, d, eps)
    out = {"dW1": np.zeros_like(W1), "db1": np.zeros(W1.shape[1]), "dW3": np.zeros_like(W3),
           "dWq": np.zeros_like(Wq), "dWk": np.zeros_like(Wk), "dWv": np.zeros_like(Wv)}
    ds_raw = np.zeros_like(s_raw)
    dd = np.zeros_like(d)
    scale = 1.0 / np.sqrt(dh)
    for h in range(H):
        rows = slice(h * dh, (h + 1) * dh)
        # Z[h] = s1[h] W3[rows]
        ds1 = dZ[h] @ W3[rows].T
        out["dW3"][rows] = s1[h].T @ dZ[h]
        # s1 = softmax(q k^T * scale) v with q, k, v = s Wq, s Wk, s Wv
        q, k, v = s[h] @ Wq[h], s[h] @ Wk[h], s[h] @ Wv[h]
        a = q @ k.T * scale
        p = np.exp(a - a.max(axis=1, keepdims=True))
        p = p / p.sum(axis=1, keepdims=True)
        dv = p.T @ ds1
        dp = ds1 @ v.T
        da = p * (dp - (dp * p).sum(axis=1, keepdims=True))
        dq = da @ k * scale
        dk = da.T @ q * scale
        out["dWq"][h] = s[h].T @ dq
        out["dWk"][h] = s[h].T @ dk
        out["dWv"][h] = s[h].T @ dv
        ds = dq @ Wq[h].T + dk @ Wk[h].T + dv @ Wv[h].T
        # s[h] = mean[h] W1[:, rows] + b1[rows]
        out["dW1"][:, rows] = mean[h].T @ ds
        out["db1"][rows] = ds.sum(axis=0)
        dmean = ds @ W1[:, rows].T
        # mean = s_raw / den where den > 0, else 0 (constant)
        live = den[h, :, 0] > 0
        ds_raw[h][live] = dmean[live] / den[h][live]
        dd[h][live] = -(dmean[live] * mean[h][live]).sum(axis=1) / den[h, live, 0]
    return ds_raw, dd, out


def dx_tile(x_tile, g_tile, W2, b2, Z, ds_raw, dd, H: int, M: int, inv_tau: float):
    """Pass B2 on one tile: (dx_tile, dW2 contribution, db2 contribution)."""
    x_tile, g_tile = _f64(x_tile), _f64(g_tile)
    N = len(x_tile)
    w = slice_weights(x_tile, W2, b2, H, M, inv_tau)
    dw = (np.einsum("nc,hmc->nhm", g_tile, _f64(Z)) + np.einsum("nc,hmc->nhm", x_tile, _f64(ds_raw))
          + _f64(dd)[None])
    dz = inv_tau * w * (dw - (w * dw).sum(axis=2, keepdims=True))
    dz2 = dz.reshape(N, H * M)
    dx = dz2 @ _f64(W2).T + np.einsum("nhm,hmc->nc", w, _f64(ds_raw))
    return dx, x_tile.T @ dz2, dz2.sum(axis=0)


def layer_backward(x, W, g, H: int, M: int, inv_tau: float, tile: int | None = None, eps: float = 0.0):
    """Gradients of sum(g * x_out) for x_out = layer_forward_fast(x, W, ...):
    dict with dx and dW2, db2, dW1, db1, dWq, dWk, dWv, dW3, db3."""
    x, g = _f64(x), _f64(g)
    N, C = x.shape
    tile = N if not tile else tile
    st = build_state(x, W, H, M, inv_tau, tile, eps)
    dZ = np.zeros((H, M, C))
    for t0 in range(0, N, max(tile, 1)):
        dZ += dZ_accumulate(x[t0:t0 + tile], g[t0:t0 + tile], W["W2"], W["b2"], H, M, inv_tau)
    ds_raw, dd, grads = token_backward(st, dZ, W, H, eps)
    grads["db3"] = g.sum(axis=0)
    dx = np.empty_like(x)
    dW2 = np.zeros(np.shape(W["W2"]))
    db2 = np.zeros(np.shape(W["b2"]))
    for t0 in range(0, N, max(tile, 1)):
        dxt, dw2t, db2t = dx_tile(x[t0:t0 + tile], g[t0:t0 + tile], W["W2"], W["b2"], st["Z"], ds_raw, dd,
                                  H, M, inv_tau)
        dx[t0:t0 + tile] = dxt
        dW2 += dw2t
        db2 += db2t
    grads.update(dx=dx, dW2=dW2, db2=db2, dZ=dZ, ds_raw=ds_raw, dd=dd)
    return grads
