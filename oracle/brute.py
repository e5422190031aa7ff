"""Brute-force loop form of the Physics-Attention layer, for tiny inputs.

TEST INFRASTRUCTURE (see ``oracle/physics_attention.py``).  Plain Python
loops over points, heads, slices and channels with ``math.exp``; no numpy
linear algebra, so it checks the vectorised oracle independently.  Follows
Eq. (1)-(2) of section 3.1 directly: project, softmax slice weights, weighted
mean per slice, per-head attention among the slice tokens, deslice, project.
"""
from __future__ import annotations

import math


def _matvec_row(row, W, col0, ncol):
    """row [K] times columns col0..col0+ncol of W [K][*] -> list."""
    return [sum(row[k] * W[k][col0 + j] for k in range(len(row))) for j in range(ncol)]


def slice_tokens_loops(x, W, H, M, inv_tau, eps=0.0):
    """Slice weights w[i][h][m] and slice tokens s[h][m][k] of Eq. (1)-(2):
    project each point with Linear1, then take each slice's weighted mean."""
    x = [list(map(float, r)) for r in x]
    N, C = len(x), len(x[0])
    dh = C // H
    W2 = W["W2"].tolist(); b2 = W["b2"].tolist()
    W1 = W["W1"].tolist(); b1 = W["b1"].tolist()

    # slice weights w[i][h][m]
    w = []
    for i in range(N):
        wi = []
        for h in range(H):
            logit = [(sum(x[i][c] * W2[c][h * M + m] for c in range(C)) + b2[h * M + m]) * inv_tau
                     for m in range(M)]
            top = max(logit)
            e = [math.exp(v - top) for v in logit]
            z = sum(e)
            wi.append([v / z for v in e])
        w.append(wi)

    # x_proj[i][h][k] = (x W1 + b1) for head h's block
    xp = [[[v + b1[h * dh + k] for k, v in enumerate(_matvec_row(x[i], W1, h * dh, dh))]
           for h in range(H)] for i in range(N)]

    # s[h][m][k] = sum_i w x_proj / sum_i w
    s = [[[0.0] * dh for _ in range(M)] for _ in range(H)]
    for h in range(H):
        for m in range(M):
            den = sum(w[i][h][m] for i in range(N)) + eps
            for k in range(dh):
                num = sum(w[i][h][m] * xp[i][h][k] for i in range(N))
                s[h][m][k] = num / den if den > 0 else 0.0
    return w, s


def layer_forward_loops(x, W, H, M, inv_tau, eps=0.0):
    N, C = len(x), len(x[0])
    dh = C // H
    w, s = slice_tokens_loops(x, W, H, M, inv_tau, eps)
    Wq = W["Wq"].tolist(); Wk = W["Wk"].tolist(); Wv = W["Wv"].tolist()
    W3 = W["W3"].tolist(); b3 = W["b3"].tolist()

    # per-head attention among M tokens
    s1 = [[[0.0] * dh for _ in range(M)] for _ in range(H)]
    for h in range(H):
        q = [_matvec_row(s[h][m], Wq[h], 0, dh) for m in range(M)]
        kk = [_matvec_row(s[h][m], Wk[h], 0, dh) for m in range(M)]
        v = [_matvec_row(s[h][m], Wv[h], 0, dh) for m in range(M)]
        for a in range(M):
            sc = [sum(q[a][j] * kk[b][j] for j in range(dh)) / math.sqrt(dh) for b in range(M)]
            top = max(sc)
            e = [math.exp(t - top) for t in sc]
            z = sum(e)
            for j in range(dh):
                s1[h][a][j] = sum(e[b] / z * v[b][j] for b in range(M))

    # deslice then Linear3
    out = []
    for i in range(N):
        mid = [sum(w[i][h][m] * s1[h][m][k] for m in range(M)) for h in range(H) for k in range(dh)]
        out.append([sum(mid[j] * W3[j][c] for j in range(H * dh)) + b3[c] for c in range(C)])
    return out
