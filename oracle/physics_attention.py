"""Plain float64 CPU oracle for one Physics-Attention layer of Transolver-3.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline may import this module.  It shares no code with the GPU path and the
GPU path never calls it.

Notation (paper section 3): x [N, C] point features; H heads, each with M
slices; dh = C / H head width; tau the softmax temperature, passed as
``inv_tau`` = 1/tau so that 1/tau = 0 (uniform weights) is expressible.
Weights: W2 [C, H*M], b2 [H*M] (Linear2, slice logits); W1 [C, H*dh], b1
(Linear1); Wq, Wk, Wv [H, dh, dh] (token attention, no bias); W3 [H*dh, C],
b3 [C] (Linear3).  Multi-head reading: Linear2's output is split into H groups
of M logits and each group gets its own softmax; head h's tokens use columns
h*dh:(h+1)*dh of W1 and the same rows of W3; attention runs per head among
that head's M tokens with scale 1/sqrt(dh).

Two forms are given and must agree (the paper states the reordering is exact,
section 3.2, "Faster slice and deslice"):
  * ``layer_forward_orig``: project then slice, Eq. (1)-(2);
  * ``layer_forward_fast``: slice then project: the state of Eq. (3) in closed
    form over the whole mesh, then each point decoded by Eq. (5).  Eq. (4)'s
    additivity over parts of the mesh is what tiling relies on; it is a pinned
    property here, not the way the state is defined.
The reordered form is also exposed in pieces (``slice_accumulate`` for any
part of the mesh, ``token_side`` ... ``deslice``) so each GPU entry point has
a matching oracle step; ``projected_accumulate`` / ``projected_finalize`` give
the state from sums taken after Linear1 (the order of Eq. (2)), for GPU paths
that accumulate projected sums.

Parity pins: every function here is checked in ``tests/test_oracle.py``
against brute-force loops, closed forms (M = 1, 1/tau = 0, one-hot slices),
invariants (softmax rows sum to one, permutation and duplication invariance,
tiling and chunking invariance) and a library attention routine.
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# --------------------------------------------------------------------- Eq. (1)

def slice_weights(x, W2, b2, H: int, M: int, inv_tau: float) -> np.ndarray:
    """w = Softmax(Linear2(x)) per head, Eq. (1) second line -> [N, H, M].

    Logits are scaled by 1/tau before the softmax; each (point, head) row
    sums to one.  Subtracting the row maximum leaves the softmax unchanged.
    """
    x = _f64(x)
    logits = (x @ _f64(W2) + _f64(b2)).reshape(len(x), H, M) * inv_tau
    logits = logits - logits.max(axis=2, keepdims=True) if len(x) else logits
    e = np.exp(logits)
    return e / e.sum(axis=2, keepdims=True)


def token_attention(s, Wq, Wk, Wv) -> np.ndarray:
    """Attention among each head's M slice tokens: s [H, M, dh] -> s' [H, M, dh]."""
    s = _f64(s)
    H, M, dh = s.shape
    out = np.empty_like(s)
    for h in range(H):
        q = s[h] @ _f64(Wq)[h]
        k = s[h] @ _f64(Wk)[h]
        v = s[h] @ _f64(Wv)[h]
        a = q @ k.T / np.sqrt(dh)
        a = np.exp(a - a.max(axis=1, keepdims=True))
        a = a / a.sum(axis=1, keepdims=True)
        out[h] = a @ v
    return out


# ----------------------------------------------------------- Eq. (1)-(2), ORIG

def layer_forward_orig(x, W, H: int, M: int, inv_tau: float, eps: float = 0.0) -> np.ndarray:
    """Original Physics-Attention: project, slice, attend, deslice, project.

    x_proj = Linear1(x); s = (w d^-1)^T x_proj with d_jj = sum_i w_ij;
    s' = Attention(s); x_out = Linear3(w s')   (Eq. (1) and (2)).
    """
    x = _f64(x)
    N, C = x.shape
    dh = C // H
    w = slice_weights(x, W["W2"], W["b2"], H, M, inv_tau)            # [N,H,M]
    x_proj = (x @ _f64(W["W1"]) + _f64(W["b1"])).reshape(N, H, dh)   # [N,H,dh]
    d = w.sum(axis=0)                                                # [H,M]
    num = np.einsum("nhm,nhd->hmd", w, x_proj)
    den = (d + eps)[:, :, None]
    s = np.divide(num, den, out=np.zeros_like(num), where=den > 0)
    s1 = token_attention(s, W["Wq"], W["Wk"], W["Wv"])
    x_mid = np.einsum("nhm,hmd->nhd", w, s1).reshape(N, H * dh)      # w s'
    return x_mid @ _f64(W["W3"]) + _f64(W["b3"])


# --------------------------------------------- Eq. (3)-(5), Algorithm 1, FAST

def slice_accumulate(x_tile, W2, b2, H: int, M: int, inv_tau: float):
    """One tile's contribution, Eq. (4): s_raw^(t) = w^(t)T x^(t) [H, M, C] and
    d^(t) = sum_i w^(t)_i [H, M]."""
    x_tile = _f64(x_tile)
    w = slice_weights(x_tile, W2, b2, H, M, inv_tau)
    return np.einsum("nhm,nc->hmc", w, x_tile), w.sum(axis=0)


def slice_finalize(s_raw, d, W1, b1, H: int, eps: float = 0.0):
    """s = Linear1(d^-1 s_raw) per head: normalise first, then Linear1.

    The normalised mean d^-1 s_raw is the physical state of Appendix A.4; an
    empty slice (d + eps = 0) has mean zero.  Head h uses W1[:, h*dh:(h+1)*dh].
    """
    s_raw, d = _f64(s_raw), _f64(d)
    C = s_raw.shape[2]
    dh = C // H
    den = (d + eps)[:, :, None]
    mean = np.divide(s_raw, den, out=np.zeros_like(s_raw), where=den > 0)
    W1, b1 = _f64(W1), _f64(b1)
    return np.stack([mean[h] @ W1[:, h * dh:(h + 1) * dh] + b1[h * dh:(h + 1) * dh]
                     for h in range(H)])


def projected_accumulate(x_tile, W2, b2, W1, H: int, M: int, inv_tau: float):
    """One tile's contribution with Linear1 applied per point first, the order
    of Eq. (2): each point's head-h projection f_ih = x_i W1[:, h*dh:(h+1)*dh]
    (without b1) is summed with its slice weights, t^(t) = sum_i w_ih f_ih
    [H, M, dh], with d^(t) = sum_i w_i [H, M].  Linear1 is linear, so
    t = s_raw W1_h per head: the sums of Eq. (4) taken after the projection."""
    x_tile = _f64(x_tile)
    N, C = x_tile.shape
    dh = C // H
    w = slice_weights(x_tile, W2, b2, H, M, inv_tau)
    f = (x_tile @ _f64(W1)).reshape(N, H, dh)
    return np.einsum("nhm,nhj->hmj", w, f), w.sum(axis=0)


def projected_finalize(t_raw, d, b1, H: int, eps: float = 0.0):
    """s = d^-1 t + b1 per head from projected sums: the same s as
    ``slice_finalize`` (the mean commutes with the bias-free projection, and
    b1 is added once per slice token); an empty slice gives s = b1."""
    t_raw, d = _f64(t_raw), _f64(d)
    dh = t_raw.shape[2]
    den = (d + eps)[:, :, None]
    mean = np.divide(t_raw, den, out=np.zeros_like(t_raw), where=den > 0)
    return mean + _f64(b1).reshape(H, 1, dh)


def linear3_tokens(s1, W3) -> np.ndarray:
    """s'_out = Linear3(s') applied per token without the bias: Z [H, M, C].

    Head h's tokens meet rows h*dh:(h+1)*dh of W3.  The bias b3 is added once per
    point in ``deslice``: each head's slice weights sum to one, so adding it per
    token would count it H times.
    """
    s1 = _f64(s1)
    H, M, dh = s1.shape
    W3 = _f64(W3)
    return np.stack([s1[h] @ W3[h * dh:(h + 1) * dh] for h in range(H)])


def deslice(x_chunk, W2, b2, Z, b3, H: int, M: int, inv_tau: float) -> np.ndarray:
    """Full-mesh decoding, Eq. (5): w = Softmax(Linear2(x)); x_out = w s'_out + b3."""
    w = slice_weights(x_chunk, W2, b2, H, M, inv_tau)
    return np.einsum("nhm,hmc->nc", w, _f64(Z)) + _f64(b3)


def token_side(s_raw, d, W, H: int, eps: float = 0.0):
    """Eq. (3) after the sums over the mesh, and section 3.3's cached state:
    s = Linear1(d^-1 s_raw), s' = Attention(s), Z = s'_out = Linear3(s')."""
    s = slice_finalize(s_raw, d, W["W1"], W["b1"], H, eps)
    s1 = token_attention(s, W["Wq"], W["Wk"], W["Wv"])
    return {"s": s, "s1": s1, "Z": linear3_tokens(s1, W["W3"])}


def build_state(x, W, H: int, M: int, inv_tau: float, tile: int | None = None, eps: float = 0.0):
    """The physical state of Eq. (3): s_raw = w^T x and d = sum_i w_i over the
    whole mesh, then the token side.  Returns s_raw, d, s, s1 and Z (= s'_out).

    The two sums are additive over any partition of the mesh (Eq. (4)); a
    `tile` only splits the mesh into consecutive parts of that many points to
    bound the memory of w, and the parts' sums are added in order."""
    x = _f64(x)
    N, C = x.shape
    parts = [x] if not tile or N <= tile else [x[i:i + tile] for i in range(0, N, tile)]
    sums = [slice_accumulate(p, W["W2"], W["b2"], H, M, inv_tau) for p in parts]
    s_raw = sum((t[0] for t in sums), np.zeros((H, M, C)))
    d = sum((t[1] for t in sums), np.zeros((H, M)))
    return {"s_raw": s_raw, "d": d, **token_side(s_raw, d, W, H, eps)}


def layer_forward_fast(x, W, H: int, M: int, inv_tau: float, tile: int | None = None,
                       chunk: int | None = None, eps: float = 0.0) -> np.ndarray:
    """The reordered layer: the state of Eq. (3) over the whole mesh, then every
    point decoded from it by Eq. (5).  `tile` and `chunk` only bound memory
    (Eq. (4) and the point-wise decode make the result independent of them)."""
    x = _f64(x)
    Z = build_state(x, W, H, M, inv_tau, tile, eps)["Z"]
    if not chunk or len(x) <= chunk:
        return deslice(x, W["W2"], W["b2"], Z, W["b3"], H, M, inv_tau)
    return np.concatenate([deslice(x[c:c + chunk], W["W2"], W["b2"], Z, W["b3"], H, M, inv_tau)
                           for c in range(0, len(x), chunk)])
