"""Pure-Python brute force of the same definitions, for tiny shapes only.

TEST INFRASTRUCTURE ONLY.  Written independently of ``estp_oracle``: scalar
loops, ``math.exp``/``math.log`` and ``math.fsum``, the full attention
matrix of every head materialised, averaged over heads and then
column-averaged exactly as Eq. 1 reads.  It exists to pin the vectorised
oracle on small random inputs.
"""
from __future__ import annotations

import math


def _f(x) -> float:
    return float(x)


def entropy_rows(X, W):
    """[H_i] for rows of X: logits z_v = sum_k W[v][k] X[i][k], H = -sum p log p (Eq. 2)."""
    out = []
    V = len(W)
    for x in X:
        z = [math.fsum(_f(W[v][k]) * _f(x[k]) for k in range(len(x))) for v in range(V)]
        zmax = max(z)
        Z = math.fsum(math.exp(zv - zmax) for zv in z)
        H = 0.0
        terms = []
        for zv in z:
            p = math.exp(zv - zmax) / Z
            if p > 0.0:
                terms.append(-p * math.log(p))
        H = math.fsum(terms)
        out.append(H)
    return out


def importance(Q, K, lengths, scale, exclude_self=False):
    """S for one layer: Q[t][h][k], K[t][g][k] nested lists, prompts given by ``lengths`` (Eq. 1);
    ``exclude_self`` leaves the diagonal out of the column sums."""
    Hq = len(Q[0])
    Hkv = len(K[0])
    G = Hq // Hkv
    S = []
    start = 0
    for N in lengths:
        # A averaged over heads, N x N, zero above the diagonal
        Aavg = [[0.0] * N for _ in range(N)]
        for h in range(Hq):
            g = h // G
            for i in range(N):
                s = []
                for j in range(i + 1):
                    qi = Q[start + i][h]
                    kj = K[start + j][g]
                    s.append(scale * math.fsum(_f(qi[c]) * _f(kj[c]) for c in range(len(qi))))
                smax = max(s)
                den = math.fsum(math.exp(v - smax) for v in s)
                for j in range(i + 1):
                    Aavg[i][j] += math.exp(s[j] - smax) / den / Hq
        for j in range(N):
            S.append(math.fsum(Aavg[i][j] for i in range(N) if not (exclude_self and i == j)) / N)
        start += N
    return S


def fused_weights(S, H, lengths, lambda1, lambda2, alpha):
    """e_i = exp(T_i / alpha) / sum_j exp(T_j / alpha), T = lambda1 S + lambda2 H (Eq. 3, 4)."""
    e = []
    start = 0
    for N in lengths:
        T = [lambda1 * S[start + i] + lambda2 * H[start + i] for i in range(N)]
        m = max(T)
        w = [math.exp((t - m) / alpha) for t in T]
        den = math.fsum(w)
        e.extend(v / den for v in w)
        start += N
    return e


def pooled(X, e, lengths):
    """h = sum_i e_i h_i per prompt (Eq. 5)."""
    out = []
    start = 0
    d = len(X[0])
    for N in lengths:
        out.append([math.fsum(e[start + i] * _f(X[start + i][c]) for i in range(N)) for c in range(d)])
        start += N
    return out


def row_lse(Q, K, lengths, scale):
    """lse[h][t] = log sum_{j <= i} exp(scale q_i . k_j) for token t = start + i of each prompt (one layer)."""
    Hq = len(Q[0])
    G = Hq // len(K[0])
    out = [[0.0] * len(Q) for _ in range(Hq)]
    start = 0
    for N in lengths:
        for h in range(Hq):
            for i in range(N):
                s = [scale * math.fsum(_f(Q[start + i][h][c]) * _f(K[start + j][h // G][c]) for c in range(len(Q[0][0])))
                     for j in range(i + 1)]
                smax = max(s)
                out[h][start + i] = smax + math.log(math.fsum(math.exp(v - smax) for v in s))
        start += N
    return out


def importance_with_lse(Q, K, lengths, scale, lse):
    """S for one layer with attention rows exp(s_ij - lse[h][t_i]) (Eq. 1 with given row normalisers)."""
    Hq = len(Q[0])
    G = Hq // len(K[0])
    S = []
    start = 0
    for N in lengths:
        for j in range(N):
            terms = []
            for h in range(Hq):
                for i in range(j, N):
                    s = scale * math.fsum(_f(Q[start + i][h][c]) * _f(K[start + j][h // G][c]) for c in range(len(Q[0][0])))
                    terms.append(math.exp(s - lse[h][start + i]) / Hq)
            S.append(math.fsum(terms) / N)
        start += N
    return S
