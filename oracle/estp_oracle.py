"""Plain fp64 definitions of the ESTP scoring and pooling path.

TEST INFRASTRUCTURE ONLY (see the package docstring): the product path never
imports this module.

Notation follows the paper: hidden states h_i (here rows of ``X``), entropy
H_i (Eq. 2), attention importance S_j (Eq. 1), fused score T_i (Eq. 3),
pooling weights e_i (Eq. 4), pooled representation h (Eq. 5), bin
probabilities p-hat and expected length y-hat (Eq. 7).

Readings of points the paper leaves open (each is also listed with its
reason in the design notes of the repository):

* H_i is the entropy of the LM-head distribution computed from token i's own
  final-layer hidden state, for every prompt token including the last; the LM
  head is ``W @ h_i`` with no bias, scaling or cap; natural log (nats).
* A is the causal self-attention of one layer averaged over the Hq query
  heads; the diagonal A_jj is part of the sum in Eq. 1; the normaliser is the
  prompt's own length N; with several layers the per-layer S are summed.
  Scores are ``scale * q_i . k_j`` with ``scale = 1/sqrt(dh)`` on post-RoPE
  queries and keys; query head h reads key head ``h // (Hq // Hkv)``.
* Eq. 4 is read with the temperature the text names: e = softmax(T / alpha).
* ``norm="zscore"`` replaces S and H by their per-prompt z-scores before
  Eq. 3 (population std, epsilon 1e-6); ``norm="minmax"`` by
  (v - min) / (max - min + 1e-6) per prompt; ``norm="none"`` is Eq. 3 literally.
* ties (top token, bin argmax) go to the lowest index; the shortest-job-first
  order is a stable ascending sort of y-hat.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np


# ----------------------------------------------------------------------------- inputs

def widen(a) -> np.ndarray:
    """Exact float64 copy of bf16 bit patterns (uint16) or of a float array."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ----------------------------------------------------------------------------- Eq. 2

def token_entropy(X, W, row_chunk: Optional[int] = None) -> np.ndarray:
    """H_i = -sum_v P(v) log P(v), P = softmax over the vocabulary of W h_i (Eq. 2).

    ``X`` [n, d] hidden states, ``W`` [V, d] LM-head weight.  Rows are
    processed ``row_chunk`` at a time only to bound memory (default: about
    512 MiB of logits per chunk); every row sees its complete logit vector.
    """
    Xd = widen(X)
    Wd = widen(W)
    n = Xd.shape[0]
    if row_chunk is None:
        row_chunk = int(max(64, min(1024, (1 << 26) // max(1, Wd.shape[0]))))
    H = np.empty(n, dtype=np.float64)
    for r0 in range(0, n, row_chunk):
        z = Xd[r0:r0 + row_chunk] @ Wd.T                      # logits, [rows, V]
        m = z.max(axis=1, keepdims=True)
        lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))   # log of the partition sum
        logp = z - lse                                         # log P(v)
        p = np.exp(logp)
        H[r0:r0 + row_chunk] = -(p * logp).sum(axis=1)
    return H


def vocab_argmax(X, W, row_chunk: Optional[int] = None) -> np.ndarray:
    """Most probable next token of each row under Eq. 2's distribution (Section 4.2).

    P_i = softmax(W h_i) is increasing in the logit, so the mode is the index
    of the largest logit z_v = W[v] . h_i; among equal largest logits the
    lowest index.  Logits are formed exactly as in ``token_entropy`` (fp64
    products of the widened inputs).  Returns int64 [n].
    """
    Xd = widen(X)
    Wd = widen(W)
    n = Xd.shape[0]
    if row_chunk is None:
        row_chunk = int(max(64, min(1024, (1 << 26) // max(1, Wd.shape[0]))))
    out = np.empty(n, dtype=np.int64)
    for r0 in range(0, n, row_chunk):
        z = Xd[r0:r0 + row_chunk] @ Wd.T
        out[r0:r0 + row_chunk] = np.argmax(z, axis=1)     # first occurrence of the maximum
    return out


# ----------------------------------------------------------------------------- Eq. 1

def _causal_softmax_rows(s: np.ndarray, i0: int) -> np.ndarray:
    """Row-wise softmax of scores s [rows, N] for queries i0.., keys j <= i only."""
    rows, N = s.shape
    i = np.arange(i0, i0 + rows)[:, None]
    j = np.arange(N)[None, :]
    s = np.where(j <= i, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    return p / p.sum(axis=1, keepdims=True)


def attn_importance(Q, K, cu_seqlens, scale: Optional[float] = None, row_chunk: int = 2048,
                    exclude_self: bool = False, layer_weights=None) -> np.ndarray:
    """S_j = (1/N) sum_i A_ij with A the head-averaged causal attention (Eq. 1).

    ``Q`` [L, n_tok, Hq, dh] and ``K`` [L, n_tok, Hkv, dh] are post-RoPE
    queries and keys of L layers, packed over prompts by ``cu_seqlens``
    [B+1]; the result [n_tok] sums the per-layer importance, each layer
    weighted by ``layer_weights[l]`` when given.  Query rows are taken
    ``row_chunk`` at a time (the column sum over i is split into consecutive
    ranges); each attention row is complete.  ``exclude_self`` drops the
    diagonal term A_jj from the column sum (the rows themselves still include
    it): the variant reading of the paper's note on self-similarity.
    """
    Qd = widen(Q)
    Kd = widen(K)
    if Qd.ndim == 3:
        Qd, Kd = Qd[None], Kd[None]
    L, n_tok, Hq, dh = Qd.shape
    Hkv = Kd.shape[2]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    S = np.zeros(n_tok, dtype=np.float64)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        N = hi - lo
        if N <= 0:
            continue
        for l in range(L):
            colsum = np.zeros(N, dtype=np.float64)           # sum_i of the head-averaged A_ij
            for h in range(Hq):
                q = Qd[l, lo:hi, h, :]
                k = Kd[l, lo:hi, h // G, :]
                for i0 in range(0, N, row_chunk):
                    s = scale * (q[i0:i0 + row_chunk] @ k.T)
                    A = _causal_softmax_rows(s, i0)
                    if exclude_self:
                        r = np.arange(A.shape[0])
                        A[r, i0 + r] = 0.0
                    colsum += A.sum(axis=0) / Hq
            S[lo:hi] += (1.0 if layer_weights is None else float(layer_weights[l])) * colsum / N
    return S


def attn_row_lse(Q, K, cu_seqlens, scale: Optional[float] = None, row_chunk: int = 2048) -> np.ndarray:
    """Log partition sum of every causal attention row, [L, Hq, n_tok] (natural log).

    lse_{l,h,i} = log sum_{j <= i, j in i's prompt} exp(scale q_i . k_j), the
    normaliser of A_ij in Eq. 1 (Section 4.1) and what a FlashAttention-style
    prefill returns per query row.
    """
    Qd = widen(Q)
    Kd = widen(K)
    if Qd.ndim == 3:
        Qd, Kd = Qd[None], Kd[None]
    L, n_tok, Hq, dh = Qd.shape
    G = Hq // Kd.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = np.empty((L, Hq, n_tok), dtype=np.float64)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        N = hi - lo
        if N <= 0:
            continue
        j = np.arange(N)[None, :]
        for l in range(L):
            for h in range(Hq):
                q = Qd[l, lo:hi, h, :]
                k = Kd[l, lo:hi, h // G, :]
                for i0 in range(0, N, row_chunk):
                    s = scale * (q[i0:i0 + row_chunk] @ k.T)
                    i = np.arange(i0, i0 + s.shape[0])[:, None]
                    s = np.where(j <= i, s, -np.inf)
                    m = s.max(axis=1)
                    out[l, h, lo + i0:lo + i0 + s.shape[0]] = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    return out


def attn_importance_from_lse(Q, K, cu_seqlens, lse, scale: Optional[float] = None,
                             row_chunk: int = 2048, exclude_self: bool = False, layer_weights=None) -> np.ndarray:
    """S_j of Eq. 1 with row i of every head normalised by the given ``lse`` [L, Hq, n_tok]:
    A_ij = exp(scale q_i . k_j - lse_i) for j <= i, then averaged over heads,
    summed over i and divided by N as in ``attn_importance``.  With
    ``lse = attn_row_lse(...)`` the rows are the causal softmax rows and the
    result is ``attn_importance``.  ``exclude_self`` and ``layer_weights`` as there.
    """
    Qd = widen(Q)
    Kd = widen(K)
    lse = np.asarray(lse, dtype=np.float64)
    if Qd.ndim == 3:
        Qd, Kd = Qd[None], Kd[None]
        lse = lse[None] if lse.ndim == 2 else lse
    L, n_tok, Hq, dh = Qd.shape
    G = Hq // Kd.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    S = np.zeros(n_tok, dtype=np.float64)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        N = hi - lo
        if N <= 0:
            continue
        j = np.arange(N)[None, :]
        for l in range(L):
            colsum = np.zeros(N, dtype=np.float64)
            for h in range(Hq):
                q = Qd[l, lo:hi, h, :]
                k = Kd[l, lo:hi, h // G, :]
                for i0 in range(0, N, row_chunk):
                    s = scale * (q[i0:i0 + row_chunk] @ k.T)
                    i = np.arange(i0, i0 + s.shape[0])[:, None]
                    keep = (j < i) if exclude_self else (j <= i)
                    A = np.where(keep, np.exp(s - lse[l, h, lo + i0:lo + i0 + s.shape[0]][:, None]), 0.0)
                    colsum += A.sum(axis=0) / Hq
            S[lo:hi] += (1.0 if layer_weights is None else float(layer_weights[l])) * colsum / N
    return S


def attn_importance_tail(Q, K, N: int, m: int, scale: Optional[float] = None) -> np.ndarray:
    """S_j of Eq. 1 for the last ``m`` keys j = N-m .. N-1 of ONE prompt of length N.

    Only queries i >= j attend to key j under the causal mask, so these m
    values need just the last m attention rows (each row still over all of
    its i+1 keys).  ``Q`` [L, N, Hq, dh], ``K`` [L, N, Hkv, dh] hold that
    prompt alone.  Returns [m], summed over layers like ``attn_importance``.
    """
    Qd = widen(Q)
    Kd = widen(K)
    if Qd.ndim == 3:
        Qd, Kd = Qd[None], Kd[None]
    L, n, Hq, dh = Qd.shape
    if n != N or not 1 <= m <= N:
        raise ValueError("Q, K must hold exactly the prompt and 1 <= m <= N")
    G = Hq // Kd.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    i0 = N - m
    S = np.zeros(m, dtype=np.float64)
    for l in range(L):
        colsum = np.zeros(m, dtype=np.float64)
        for h in range(Hq):
            s = scale * (Qd[l, i0:, h, :] @ Kd[l, :, h // G, :].T)   # rows i0..N-1, all keys
            A = _causal_softmax_rows(s, i0)
            colsum += A[:, i0:].sum(axis=0) / Hq
        S += colsum / N
    return S


def attn_importance_keys(Q, K, N: int, keys, scale: Optional[float] = None, heads=None,
                         row_chunk: int = 256) -> np.ndarray:
    """S_j of Eq. 1 for the keys ``keys`` (any indices 0 <= j < N) of ONE prompt of length N.

    Key j receives attention from the queries i >= j only, so every row
    i >= min(keys) is formed in full (all of its i+1 causal scores, its own
    softmax normaliser) and its entries at the requested keys are added to
    their column sums.  ``Q`` [L, N, Hq, dh] and ``K`` [L, N, Hkv, dh] hold
    that prompt alone.  ``heads`` restricts the head average of Eq. 1 to a
    subset of the query heads (each term still divided by Hq), so that the
    sums over a partition of the heads add up to S; default all heads.
    Returns [len(keys)], summed over layers like ``attn_importance``.  Inputs
    are widened one (layer, head) at a time, so long prompts stay in memory.
    """
    Q = np.asarray(Q)
    K = np.asarray(K)
    if Q.ndim == 3:
        Q, K = Q[None], K[None]
    L, n, Hq, dh = Q.shape
    keys = np.asarray(keys, dtype=np.int64)
    if n != N or keys.size == 0 or keys.min() < 0 or keys.max() >= N:
        raise ValueError("Q, K must hold exactly the prompt and every key must lie in [0, N)")
    G = Hq // K.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    heads = range(Hq) if heads is None else heads
    first = int(keys.min())
    S = np.zeros(keys.size, dtype=np.float64)
    for l in range(L):
        colsum = np.zeros(keys.size, dtype=np.float64)
        for h in heads:
            q = widen(Q[l, :, h, :])
            k = widen(K[l, :, h // G, :])
            for i0 in range(first, N, row_chunk):
                i1 = min(N, i0 + row_chunk)
                s = scale * (q[i0:i1] @ k[:i1].T)                # rows i0..i1-1, keys 0..i1-1
                A = _causal_softmax_rows(s, i0)
                colsum += _gather_cols(A, keys, i1) / Hq
        S += colsum / N
    return S


def _gather_cols(A: np.ndarray, keys: np.ndarray, width: int) -> np.ndarray:
    """Column sums of A [rows, width] at the given key indices; keys at or past ``width`` are 0."""
    out = np.zeros(keys.size, dtype=np.float64)
    inside = keys < width
    out[inside] = A[:, keys[inside]].sum(axis=0)
    return out


# ----------------------------------------------------------------------------- Eq. 3, 4

def _zscore(v: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    return (v - v.mean()) / (v.std() + eps)


def _minmax(v: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    return (v - v.min()) / (v.max() - v.min() + eps)


def combine_weights(S, H, cu_seqlens, lambda1: float, lambda2: float, alpha: float = 1.0,
                    norm: str = "none"):
    """T_i = lambda1 S_i + lambda2 H_i (Eq. 3); e = softmax over the prompt of T / alpha (Eq. 4).

    Returns ``(e [n_tok], top [B])`` where ``top[b]`` is the global index of
    the prompt's largest weight (lowest index among ties).
    """
    if not alpha > 0:
        raise ValueError("alpha must be positive")
    S = np.asarray(S, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    e = np.empty_like(S)
    top = np.empty(len(cu) - 1, dtype=np.int64)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        s, h = S[lo:hi], H[lo:hi]
        if norm == "zscore":
            s, h = _zscore(s), _zscore(h)
        elif norm == "minmax":
            s, h = _minmax(s), _minmax(h)
        elif norm != "none":
            raise ValueError(norm)
        T = lambda1 * s + lambda2 * h
        u = T / alpha
        w = np.exp(u - u.max())
        e[lo:hi] = w / w.sum()
        top[b] = lo + int(np.argmax(e[lo:hi]))
    return e, top


# ----------------------------------------------------------------------------- Eq. 5

def pool(X, e, cu_seqlens) -> np.ndarray:
    """h = sum_i e_i h_i over each prompt's tokens (Eq. 5); returns [B, d]."""
    Xd = widen(X)
    e = np.asarray(e, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = np.zeros((len(cu) - 1, Xd.shape[1]), dtype=np.float64)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        out[b] = e[lo:hi] @ Xd[lo:hi]
    return out


# ----------------------------------------------------------------------------- length head, Eq. 7

def _act(a: np.ndarray, act: str) -> np.ndarray:
    if act == "relu":
        return np.maximum(a, 0.0)
    if act == "gelu_tanh":
        return 0.5 * a * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (a + 0.044715 * a ** 3)))
    raise ValueError(act)


def predict(pooled, W1, b1, W2, b2, centres=None, act: str = "relu"):
    """MLP length head on the pooled vectors.

    ``o = W2 act(W1 h + b1) + b2``.  With one output (K = 1) y-hat is ``o``
    (direct regression); with K > 1 bins, p-hat = softmax(o) and
    y-hat = sum_k p-hat_k c_k (Eq. 7), and ``bin`` is the argmax of p-hat.
    ``order`` lists the prompts by ascending y-hat, ties by index: the
    shortest-job-first order of Section 5.4.
    Returns ``(yhat [B], bin [B] or None, order [B])``.
    """
    h = np.asarray(pooled, dtype=np.float64)
    W1 = np.asarray(W1, dtype=np.float64)
    W2 = np.asarray(W2, dtype=np.float64)
    b1 = np.zeros(W1.shape[0]) if b1 is None else np.asarray(b1, dtype=np.float64)
    b2 = np.zeros(W2.shape[0]) if b2 is None else np.asarray(b2, dtype=np.float64)
    a = _act(h @ W1.T + b1, act)
    o = a @ W2.T + b2
    K = W2.shape[0]
    if K == 1:
        yhat = o[:, 0]
        bins = None
    else:
        c = np.asarray(centres, dtype=np.float64)
        z = np.exp(o - o.max(axis=1, keepdims=True))
        phat = z / z.sum(axis=1, keepdims=True)
        yhat = phat @ c
        bins = np.argmax(phat, axis=1)
    order = np.argsort(yhat, kind="stable")
    return yhat, bins, order


# ----------------------------------------------------------------------------- Eq. 6, 8

def soft_labels(i: int, K: int) -> np.ndarray:
    """p_j = exp(-|j - i|) / sum_k exp(-|k - i|) over the K bins (Eq. 6)."""
    j = np.arange(K)
    w = np.exp(-np.abs(j - i).astype(np.float64))
    return w / w.sum()


def length_loss(p, phat, y, yhat, lambda3: float) -> float:
    """lambda3 * CE(p, p-hat) + (1 - lambda3) * MSE(y, y-hat), batch means (Eq. 8)."""
    p = np.asarray(p, dtype=np.float64)
    phat = np.asarray(phat, dtype=np.float64)
    ce = -(p * np.log(phat)).sum(axis=-1).mean()
    mse = np.mean((np.asarray(y, dtype=np.float64) - np.asarray(yhat, dtype=np.float64)) ** 2)
    return float(lambda3 * ce + (1.0 - lambda3) * mse)


# ----------------------------------------------------------------------------- training the head

def length_bin(y, edges) -> np.ndarray:
    """Index i of the bin [edges[i], edges[i+1]) holding each length; below the first
    edge -> 0, at or above the last -> K-1 (K = len(edges) - 1).  The ground-truth bin
    of Eq. 6."""
    e = np.asarray(edges, dtype=np.float64)
    K = len(e) - 1
    i = np.searchsorted(e[1:K], np.asarray(y, dtype=np.float64), side="right")
    return np.clip(i, 0, K - 1)


def _act_grad(a: np.ndarray, act: str) -> np.ndarray:
    """d act(a) / d a."""
    if act == "relu":
        return (a > 0.0).astype(np.float64)
    if act == "gelu_tanh":
        k = math.sqrt(2.0 / math.pi)
        u = k * (a + 0.044715 * a ** 3)
        t = np.tanh(u)
        return 0.5 * (1.0 + t) + 0.5 * a * (1.0 - t * t) * k * (1.0 + 3 * 0.044715 * a * a)
    raise ValueError(act)


def head_loss_and_grads(pooled, y, edges, centres, W1, b1, W2, b2, lambda3: float, act: str = "relu"):
    """Eq. 8 loss of the K-bin head (Section 4.3) on one batch and its gradients.

    Forward: a = act(W1 h + b1), o = W2 a + b2, p-hat = softmax(o), y-hat = sum_k p-hat_k c_k
    (Eq. 7); target p = Eq. 6 soft labels around the true bin; loss = lambda3 CE(p, p-hat)
    + (1 - lambda3) (y - y-hat)^2, both averaged over the batch.  Gradients by the chain rule,
    written out layer by layer.  Returns ``(loss, {"W1", "b1", "W2", "b2"})``.
    """
    h = np.asarray(pooled, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    c = np.asarray(centres, dtype=np.float64)
    W1, b1, W2, b2 = (np.asarray(t, dtype=np.float64) for t in (W1, b1, W2, b2))
    B, K = h.shape[0], W2.shape[0]
    z = h @ W1.T + b1
    a = _act(z, act)
    o = a @ W2.T + b2
    lse = o.max(axis=1, keepdims=True) + np.log(np.exp(o - o.max(axis=1, keepdims=True)).sum(axis=1, keepdims=True))
    phat = np.exp(o - lse)
    yhat = phat @ c
    p = np.stack([soft_labels(int(i), K) for i in length_bin(y, edges)])
    loss = length_loss(p, phat, y, yhat, lambda3)
    # dL/do: cross-entropy of a softmax, and the squared error through the expectation
    d_ce = phat - p
    d_mse = (-2.0 * (y - yhat))[:, None] * phat * (c[None, :] - yhat[:, None])
    do = (lambda3 * d_ce + (1.0 - lambda3) * d_mse) / B
    g = {"W2": do.T @ a, "b2": do.sum(axis=0)}
    dz = (do @ W2) * _act_grad(z, act)
    g["W1"] = dz.T @ h
    g["b1"] = dz.sum(axis=0)
    return loss, g


def adamw_step(theta, grad, m, v, t: int, lr: float, beta1: float, beta2: float, eps: float,
               weight_decay: float):
    """One AdamW step (decoupled weight decay), as the paper's optimiser (Section 5.1):
    theta <- theta (1 - lr wd); m, v <- moment updates; theta <- theta - lr m_hat / (sqrt(v_hat) + eps)
    with bias-corrected m_hat = m / (1 - beta1^t), v_hat = v / (1 - beta2^t).
    Returns ``(theta, m, v)`` (new arrays)."""
    theta = np.asarray(theta, dtype=np.float64) * (1.0 - lr * weight_decay)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * grad
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * grad * grad
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    return theta - lr * mhat / (np.sqrt(vhat) + eps), m, v


def head_train_step(pooled, y, edges, centres, params, m, v, t: int, lambda3: float, lr: float,
                    beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.01,
                    act: str = "relu"):
    """One training step of the length head: Eq. 8 loss and gradients at ``params``
    (dict W1, b1, W2, b2), then AdamW on every tensor.  ``m``, ``v`` are dicts of the same
    shapes.  Returns ``(loss, grads, params, m, v)`` with the updated dicts."""
    loss, g = head_loss_and_grads(pooled, y, edges, centres, params["W1"], params["b1"], params["W2"],
                                  params["b2"], lambda3, act)
    P, M, Vv = {}, {}, {}
    for k in ("W1", "b1", "W2", "b2"):
        P[k], M[k], Vv[k] = adamw_step(params[k], g[k], m[k], v[k], t, lr, beta1, beta2, eps, weight_decay)
    return loss, g, P, M, Vv


# ----------------------------------------------------------------------------- analyses on the outputs

def _rank_sets(v: np.ndarray, frac_low: float, frac_high: float):
    """Token sets of one prompt by rank of v (ascending, ties by lower index first): the
    floor(frac_low N) lowest and the floor(frac_high N) highest."""
    N = len(v)
    order = np.argsort(np.asarray(v, dtype=np.float64), kind="stable")
    nl, nh = int(math.floor(frac_low * N)), int(math.floor(frac_high * N))
    low = np.zeros(N, dtype=bool)
    high = np.zeros(N, dtype=bool)
    low[order[:nl]] = True
    high[order[N - nh:]] = True
    return low, high


def misalignment_counts(H, S, cu_seqlens, frac_low: float = 0.4, frac_high: float = 0.4) -> np.ndarray:
    """Entropy-semantics misalignment of each prompt (the diagnostic behind Fig. 1b, Section 1):
    tokens are split by rank within the prompt into the top ``frac_high`` and the bottom
    ``frac_low`` of H and of S.  Returns int64 [B, 4]: (#high-H, #high-H that are low-S,
    #low-H, #low-H that are high-S); the two misalignment ratios are columns 1/0 and 3/2."""
    H = np.asarray(H, dtype=np.float64)
    S = np.asarray(S, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = np.zeros((len(cu) - 1, 4), dtype=np.int64)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        lowH, highH = _rank_sets(H[lo:hi], frac_low, frac_high)
        lowS, highS = _rank_sets(S[lo:hi], frac_low, frac_high)
        out[b] = [highH.sum(), (highH & lowS).sum(), lowH.sum(), (lowH & highS).sum()]
    return out


def sjf_padding(lengths, order, batch: int):
    """Static batches of ``batch`` requests taken in ``order`` (e.g. the shortest-job-first order
    of the predicted lengths, Section 5.4); each batch runs for its longest true length.
    Returns ``(padded, useful, jct_sum)`` as integers: padded tokens sum_batches
    (size * max - sum), useful tokens sum y, and the sum over requests of the completion time
    start(batch) + y_i with batches run back to back.  Padding ratio = padded / useful;
    mean JCT = jct_sum / B."""
    y = np.asarray(lengths, dtype=np.int64)
    order = np.arange(len(y)) if order is None else np.asarray(order, dtype=np.int64)
    padded = useful = jct = 0
    start = 0
    for k0 in range(0, len(order), batch):
        members = y[order[k0:k0 + batch]]
        mx = int(members.max())
        padded += len(members) * mx - int(members.sum())
        useful += int(members.sum())
        jct += len(members) * start + int(members.sum())
        start += mx
    return padded, useful, jct


# ----------------------------------------------------------------------------- whole path

def run_path(X, W, Q, K, cu_seqlens, lambda1: float, lambda2: float, alpha: float = 1.0,
             norm: str = "none", head: Optional[Sequence] = None, act: str = "relu",
             scale: Optional[float] = None):
    """Entropy -> importance -> fused weights -> pooled vectors -> length head."""
    H = token_entropy(X, W)
    S = attn_importance(Q, K, cu_seqlens, scale)
    e, top = combine_weights(S, H, cu_seqlens, lambda1, lambda2, alpha, norm)
    h = pool(X, e, cu_seqlens)
    out = {"H": H, "S": S, "e": e, "top": top, "pooled": h}
    if head is not None:
        W1, b1, W2, b2, centres = head
        out["yhat"], out["bin"], out["order"] = predict(h, W1, b1, W2, b2, centres, act)
    return out
