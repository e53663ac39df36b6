"""Planted mistakes in the oracle must be caught by the pins.

Each mutant is the oracle's function with one plausible slip (a dropped
term, a wrong sign, index or normaliser, a transposed operand).  For every
mutant at least one pin of ``test_oracle_pins`` has to fail; this is what
makes the pins evidence for the oracle rather than a restatement of it.
"""
import math

import numpy as np
import pytest

from oracle import estp_oracle as O
from tests import test_oracle_pins as P


def _fails_some(pins, fn):
    for pin in pins:
        try:
            with np.errstate(all="ignore"):
                pin(fn)
        except Exception:
            return True
    return False


# ---------------------------------------------------------------------------- entropy mutants

def _entropy_with(logp_fn, reduce_fn=None):
    def token_entropy(X, W, row_chunk=64):
        Xd, Wd = O.widen(X), O.widen(W)
        z = Xd @ Wd.T
        logp = logp_fn(z)
        p = np.exp(logp)
        return reduce_fn(p, logp) if reduce_fn else -(p * logp).sum(axis=1)
    return token_entropy


def _lse(z, axis=1):
    m = z.max(axis=axis, keepdims=True)
    return m + np.log(np.exp(z - m).sum(axis=axis, keepdims=True))


ENTROPY_MUTANTS = {
    "sign_flipped": _entropy_with(lambda z: z - _lse(z), lambda p, lp: (p * lp).sum(axis=1)),
    "log2": _entropy_with(lambda z: z - _lse(z), lambda p, lp: -(p * lp).sum(axis=1) / math.log(2)),
    "dropped_log_partition": _entropy_with(lambda z: z - z.max(axis=1, keepdims=True)),
    "normalised_over_tokens": _entropy_with(lambda z: z - _lse(z, axis=0)),
    "previous_row": lambda X, W, row_chunk=64: np.roll(O.token_entropy(X, W), 1),
    "missing_p_factor": _entropy_with(lambda z: z - _lse(z), lambda p, lp: -lp.mean(axis=1)),
}


@pytest.mark.parametrize("name", list(ENTROPY_MUTANTS))
def test_entropy_mutant_caught(name):
    assert _fails_some(P.ENTROPY_PINS, ENTROPY_MUTANTS[name]), name


# ---------------------------------------------------------------------------- importance mutants

def _importance_mutant(kind):
    def attn_importance(Q, K, cu_seqlens, scale=None, row_chunk=2048):
        Qd, Kd = O.widen(Q), O.widen(K)
        if Qd.ndim == 3:
            Qd, Kd = Qd[None], Kd[None]
        L, n, Hq, dh = Qd.shape
        Hkv = Kd.shape[2]
        G = Hq // Hkv
        sc = 1.0 / math.sqrt(dh) if scale is None else scale
        if kind == "no_scale":
            sc = 1.0
        cu = np.asarray(cu_seqlens, dtype=np.int64)
        S = np.zeros(n)
        for b in range(len(cu) - 1):
            lo, hi = int(cu[b]), int(cu[b + 1]); N = hi - lo
            for l in range(L):
                Aavg = np.zeros((N, N))
                for h in range(Hq):
                    g = h % Hkv if kind == "gqa_modulo" else h // G
                    s = sc * Qd[l, lo:hi, h] @ Kd[l, lo:hi, g].T
                    i = np.arange(N)[:, None]; j = np.arange(N)[None, :]
                    if kind != "no_causal_mask":
                        s = np.where(j <= i, s, -np.inf)
                    if kind == "no_diagonal" and N > 1:
                        s = np.where((i == j) & (i > 0), -np.inf, s)
                    A = np.exp(s - s.max(axis=1, keepdims=True))
                    A /= A.sum(axis=1, keepdims=True)
                    Aavg += A / (Hkv if kind == "divide_by_hkv" else Hq)
                col = Aavg.sum(axis=1) if kind == "row_sums" else Aavg.sum(axis=0)
                if kind == "count_normaliser":
                    col = col / (N - np.arange(N))
                else:
                    col = col / N
                S[lo:hi] += col / (L if kind == "layer_mean" else 1)
        return S
    return attn_importance


IMPORTANCE_MUTANTS = ["row_sums", "no_causal_mask", "count_normaliser", "no_diagonal", "gqa_modulo",
                      "layer_mean", "no_scale", "divide_by_hkv"]


@pytest.mark.parametrize("kind", IMPORTANCE_MUTANTS)
def test_importance_mutant_caught(kind):
    assert _fails_some(P.IMPORTANCE_PINS, _importance_mutant(kind)), kind


def test_importance_mutant_control():
    # the mutant scaffold with no mutation passes every pin (so failures above come from the slips)
    for pin in P.IMPORTANCE_PINS:
        pin(_importance_mutant("none"))


# ---------------------------------------------------------------------------- combine mutants

def _combine_mutant(kind):
    def combine_weights(S, H, cu_seqlens, lambda1, lambda2, alpha=1.0, norm="none"):
        S = np.asarray(S, float); H = np.asarray(H, float)
        cu = np.asarray(cu_seqlens, dtype=np.int64)
        if kind == "swapped_lambdas":
            lambda1, lambda2 = lambda2, lambda1
        e = np.empty_like(S); top = np.empty(len(cu) - 1, dtype=np.int64)
        if kind == "batch_softmax":
            T = lambda1 * S + lambda2 * H
            w = np.exp(T / alpha - (T / alpha).max()); e = w / w.sum()
            for b in range(len(cu) - 1):
                top[b] = cu[b] + int(np.argmax(e[cu[b]:cu[b + 1]]))
            return e, top
        for b in range(len(cu) - 1):
            lo, hi = int(cu[b]), int(cu[b + 1])
            s, h = S[lo:hi], H[lo:hi]
            if norm == "zscore":
                s = (s - s.mean()) / (s.std() + 1e-6); h = (h - h.mean()) / (h.std() + 1e-6)
            T = lambda1 * s + lambda2 * h
            u = {"no_alpha": T, "alpha_multiplies": T * alpha}.get(kind, T / alpha)
            w = np.exp(u - u.max())
            e[lo:hi] = w / w.sum() if kind != "unnormalised" else w
            top[b] = lo + int(np.argmax(e[lo:hi]))
        return e, top
    return combine_weights


@pytest.mark.parametrize("kind", ["swapped_lambdas", "batch_softmax", "no_alpha", "alpha_multiplies", "unnormalised"])
def test_combine_mutant_caught(kind):
    assert _fails_some(P.COMBINE_PINS, _combine_mutant(kind)), kind


# ---------------------------------------------------------------------------- pool and predict mutants

def _pool_reversed(X, e, cu_seqlens):
    Xd = O.widen(X); cu = np.asarray(cu_seqlens, dtype=np.int64)
    return np.stack([np.asarray(e)[cu[b]:cu[b + 1]][::-1] @ Xd[cu[b]:cu[b + 1]] for b in range(len(cu) - 1)])


def _pool_mean(X, e, cu_seqlens):
    Xd = O.widen(X); cu = np.asarray(cu_seqlens, dtype=np.int64)
    return np.stack([Xd[cu[b]:cu[b + 1]].mean(0) for b in range(len(cu) - 1)])


def _pool_batch(X, e, cu_seqlens):
    Xd = O.widen(X); cu = np.asarray(cu_seqlens, dtype=np.int64)
    tot = np.asarray(e) @ Xd
    return np.stack([tot for _ in range(len(cu) - 1)])


@pytest.mark.parametrize("fn", [_pool_reversed, _pool_mean, _pool_batch], ids=lambda f: f.__name__)
def test_pool_mutant_caught(fn):
    assert _fails_some(P.POOL_PINS, fn)


def _predict_mutant(kind):
    def predict(pooled, W1, b1, W2, b2, centres=None, act="relu"):
        y, bins, order = O.predict(pooled, W1, b1, W2, b2, centres, act)
        if kind == "descending":
            order = np.argsort(-y, kind="stable")
        elif kind == "ties_reversed":
            order = np.lexsort((-np.arange(len(y)), y))
        elif kind == "argmin_bin" and bins is not None:
            h = np.asarray(pooled, float); a = np.maximum(h @ np.asarray(W1, float).T + (0 if b1 is None else b1), 0)
            o = a @ np.asarray(W2, float).T + (0 if b2 is None else b2)
            bins = np.argmin(o, axis=1)
        elif kind == "no_softmax" and centres is not None and np.asarray(W2).shape[0] > 1:
            h = np.asarray(pooled, float); a = np.maximum(h @ np.asarray(W1, float).T + (0 if b1 is None else b1), 0)
            o = a @ np.asarray(W2, float).T + (0 if b2 is None else b2)
            y = o @ np.asarray(centres, float)
        elif kind == "no_activation":
            h = np.asarray(pooled, float)
            o = (h @ np.asarray(W1, float).T + (0 if b1 is None else b1)) @ np.asarray(W2, float).T + (0 if b2 is None else b2)
            if o.shape[1] == 1:
                y = o[:, 0]
        return y, bins, order
    return predict


@pytest.mark.parametrize("kind", ["descending", "ties_reversed", "argmin_bin", "no_softmax", "no_activation"])
def test_predict_mutant_caught(kind):
    assert _fails_some(P.PREDICT_PINS, _predict_mutant(kind)), kind
