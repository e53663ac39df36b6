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


# ---------------------------------------------------------------------------- next-token mode mutants

def _argmax_mutant(kind):
    def vocab_argmax(X, W, row_chunk=None):
        z = O.widen(X) @ O.widen(W).T
        if kind == "last_of_ties":
            return z.shape[1] - 1 - np.argmax(z[:, ::-1], axis=1)
        if kind == "argmin":
            return np.argmin(z, axis=1)
        if kind == "off_by_one":
            return np.argmax(z, axis=1) + 1
        if kind == "mode_of_previous_row":
            return np.roll(np.argmax(z, axis=1), 1)
        if kind == "argmax_of_weight_norm":
            return np.repeat(np.argmax(np.abs(O.widen(W)).sum(axis=1)), z.shape[0])
        return np.argmax(z, axis=1)
    return vocab_argmax


@pytest.mark.parametrize("kind", ["last_of_ties", "argmin", "off_by_one", "mode_of_previous_row",
                                  "argmax_of_weight_norm"])
def test_argmax_mutant_caught(kind):
    assert _fails_some(P.ARGMAX_PINS, _argmax_mutant(kind)), kind


def test_argmax_mutant_control():
    for pin in P.ARGMAX_PINS:
        pin(_argmax_mutant("none"))


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
                if kind == "zscore_ddof1":
                    s = (s - s.mean()) / (s.std(ddof=1) + 1e-6); h = (h - h.mean()) / (h.std(ddof=1) + 1e-6)
                elif kind == "zscore_eps_in_sqrt":
                    s = (s - s.mean()) / np.sqrt(s.var() + 1e-6); h = (h - h.mean()) / np.sqrt(h.var() + 1e-6)
                else:
                    s = (s - s.mean()) / (s.std() + 1e-6); h = (h - h.mean()) / (h.std() + 1e-6)
            T = lambda1 * s + lambda2 * h
            u = {"no_alpha": T, "alpha_multiplies": T * alpha}.get(kind, T / alpha)
            w = np.exp(u - u.max())
            e[lo:hi] = w / w.sum() if kind != "unnormalised" else w
            top[b] = lo + int(np.argmax(e[lo:hi]))
        return e, top
    return combine_weights


@pytest.mark.parametrize("kind", ["swapped_lambdas", "batch_softmax", "no_alpha", "alpha_multiplies", "unnormalised",
                                  "zscore_ddof1", "zscore_eps_in_sqrt"])
def test_combine_mutant_caught(kind):
    assert _fails_some(P.COMBINE_PINS, _combine_mutant(kind)), kind


def test_combine_mutant_control():
    for pin in P.COMBINE_PINS:
        pin(_combine_mutant("none"))


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
        elif kind == "gelu_erf" and act == "gelu_tanh":
            h = np.asarray(pooled, float)
            z = h @ np.asarray(W1, float).T + (0 if b1 is None else b1)
            a = z * 0.5 * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
            o = a @ np.asarray(W2, float).T + (0 if b2 is None else b2)
            if o.shape[1] == 1:
                y = o[:, 0]
                order = np.argsort(y, kind="stable")
        elif kind == "no_activation":
            h = np.asarray(pooled, float)
            o = (h @ np.asarray(W1, float).T + (0 if b1 is None else b1)) @ np.asarray(W2, float).T + (0 if b2 is None else b2)
            if o.shape[1] == 1:
                y = o[:, 0]
        return y, bins, order
    return predict


@pytest.mark.parametrize("kind", ["descending", "ties_reversed", "argmin_bin", "no_softmax", "no_activation",
                                  "gelu_erf"])
def test_predict_mutant_caught(kind):
    assert _fails_some(P.PREDICT_PINS, _predict_mutant(kind)), kind


# ---------------------------------------------------------------------------- mutants of the later rows
# Each mutant replaces one oracle function (as the pins reach it, through the package) with a
# plausible slip; at least one of the listed pins must then fail.

import oracle  # noqa: E402


def _row_lse_excl_diag(Q, K, cu, scale=None, row_chunk=2048):
    Qd, Kd = O.widen(Q), O.widen(K)
    L, n, Hq, dh = Qd.shape
    scale = 1 / math.sqrt(dh) if scale is None else scale
    out = np.full((L, Hq, n), -np.inf)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        for l in range(L):
            for h in range(Hq):
                s = scale * Qd[l, lo:hi, h] @ Kd[l, lo:hi, h // (Hq // Kd.shape[2])].T
                s = np.where(np.arange(hi - lo)[None, :] < np.arange(hi - lo)[:, None], s, -np.inf)
                m = s.max(axis=1)
                with np.errstate(invalid="ignore"):
                    out[l, h, lo:hi] = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    return out


def _keys_mutant(kind):
    def f(Q, K, N, keys, scale=None, heads=None, row_chunk=256):
        Qd, Kd = O.widen(Q), O.widen(K)
        if Qd.ndim == 3:
            Qd, Kd = Qd[None], Kd[None]
        L, n, Hq, dh = Qd.shape
        keys = np.asarray(keys, dtype=np.int64)
        sc = 1 / math.sqrt(dh) if scale is None else scale
        G = Hq // Kd.shape[2]
        first = int(keys.max()) if kind == "rows_from_last_key" else int(keys.min())
        S = np.zeros(keys.size)
        for l in range(L):
            for h in (range(Hq) if heads is None else heads):
                for i0 in range(first, N, row_chunk):
                    i1 = min(N, i0 + row_chunk)
                    s = sc * Qd[l, i0:i1, h] @ Kd[l, :i1, h // G].T
                    if kind != "not_causal_in_chunk":
                        s = np.where(np.arange(i1)[None, :] <= np.arange(i0, i1)[:, None], s, -np.inf)
                    A = np.exp(s - s.max(axis=1, keepdims=True)); A /= A.sum(axis=1, keepdims=True)
                    inside = keys < i1
                    S[inside] += A[:, keys[inside]].sum(axis=0) / Hq
        norm = (N - keys) if kind == "per_key_count" else N
        return S / norm
    return f


def _head_mutant(kind):
    def f(pooled, y, edges, centres, W1, b1, W2, b2, lambda3, act="relu"):
        h = np.asarray(pooled, dtype=np.float64); y = np.asarray(y, dtype=np.float64)
        c = np.asarray(centres, dtype=np.float64)
        W1, b1, W2, b2 = (np.asarray(t, dtype=np.float64) for t in (W1, b1, W2, b2))
        B, K = h.shape[0], W2.shape[0]
        z = h @ W1.T + b1
        a = O._act(z, act)
        o = a @ W2.T + b2
        lse = np.log(np.exp(o - o.max(axis=1, keepdims=True)).sum(axis=1, keepdims=True)) + o.max(axis=1, keepdims=True)
        ph = np.exp(o - lse)
        yh = ph @ c
        bins = O.length_bin(y, edges)
        if kind == "hard_labels":
            p = np.eye(K)[bins]
        else:
            p = np.stack([O.soft_labels(int(i), K) for i in bins])
        loss = O.length_loss(p, ph, y, yh, lambda3)
        sgn = 2.0 if kind == "mse_grad_sign" else -2.0
        do = lambda3 * (ph - p) + (1 - lambda3) * (sgn * (y - yh))[:, None] * ph * (c[None, :] - yh[:, None])
        if kind != "no_batch_mean":
            do = do / B
        g = {"W2": do.T @ (z if kind == "w2_grad_from_z" else a), "b2": do.sum(axis=0)}
        dz = (do @ W2) * O._act_grad(a if kind == "act_grad_of_output" else z, act)
        g["W1"] = dz.T @ h
        g["b1"] = dz.sum(axis=0)
        return loss, g
    return f


def _adamw_mutant(kind):
    def f(theta, grad, m, v, t, lr, beta1, beta2, eps, weight_decay):
        theta = np.asarray(theta, dtype=np.float64)
        g = grad + weight_decay * theta if kind == "coupled_decay" else grad
        th = theta if kind == "coupled_decay" else theta * (1 - lr * weight_decay)
        m = beta1 * np.asarray(m, dtype=np.float64) + (1 - beta1) * g
        v = beta2 * np.asarray(v, dtype=np.float64) + (1 - beta2) * g * g
        mh = m if kind == "no_bias_correction" else m / (1 - beta1 ** t)
        vh = v if kind == "no_bias_correction" else v / (1 - beta2 ** t)
        den = np.sqrt(vh + eps) if kind == "eps_inside_sqrt" else np.sqrt(vh) + eps
        return th - lr * mh / den, m, v
    return f


def _misalignment_mutant(kind):
    def f(H, S, cu, frac_low=0.4, frac_high=0.4):
        out = np.zeros((len(cu) - 1, 4), dtype=np.int64)
        for b in range(len(cu) - 1):
            lo, hi = int(cu[b]), int(cu[b + 1])
            sets = []
            for v in (np.asarray(H, float)[lo:hi], np.asarray(S, float)[lo:hi]):
                N = len(v)
                if kind == "ties_by_higher_index":
                    order = np.lexsort((-np.arange(N), v))
                else:
                    order = np.argsort(v, kind="stable")
                rnd = math.ceil if kind == "ceil_counts" else math.floor
                nl, nh = int(rnd(frac_low * N)), int(rnd(frac_high * N))
                low = np.zeros(N, bool); high = np.zeros(N, bool)
                low[order[:nl]] = True; high[order[N - nh:]] = True
                sets.append((high, low) if kind == "low_high_swapped" else (low, high))
            (lowH, highH), (lowS, highS) = sets
            out[b] = [highH.sum(), (highH & lowS).sum(), lowH.sum(), (lowH & highS).sum()]
        return out
    return f


def _sjf_jct_uses_max(lengths, order, batch):
    y = np.asarray(lengths, dtype=np.int64)
    order = np.arange(len(y)) if order is None else np.asarray(order)
    padded = useful = jct = start = 0
    for k0 in range(0, len(order), batch):
        mem = y[order[k0:k0 + batch]]
        mx = int(mem.max())
        padded += len(mem) * mx - int(mem.sum()); useful += int(mem.sum())
        jct += len(mem) * (start + mx)
        start += mx
    return padded, useful, jct


LATER_MUTANTS = {
    "row_lse_excludes_diagonal": ("attn_row_lse", _row_lse_excl_diag,
                                  [P.test_row_lse_bruteforce, P.test_row_lse_closed_forms]),
    "row_lse_ignores_scale": ("attn_row_lse", lambda Q, K, cu, scale=None, row_chunk=2048: O.attn_row_lse(Q, K, cu),
                              [P.test_row_lse_bruteforce, P.test_row_lse_closed_forms]),
    "from_lse_ignores_given_lse": ("attn_importance_from_lse",
                                   lambda Q, K, cu, lse, scale=None, row_chunk=2048, exclude_self=False,
                                   layer_weights=None: O.attn_importance(Q, K, cu, scale, exclude_self=exclude_self,
                                                                         layer_weights=layer_weights),
                                   [P.test_importance_from_lse_bruteforce_and_identity]),
    "keys_rows_from_last_key": ("attn_importance_keys", _keys_mutant("rows_from_last_key"),
                                [P.test_importance_keys_match_whole_prompt, P.test_importance_keys_harmonic_and_bruteforce]),
    "keys_rows_not_causal_in_chunk": ("attn_importance_keys", _keys_mutant("not_causal_in_chunk"),
                                      [P.test_importance_keys_match_whole_prompt,
                                       P.test_importance_keys_harmonic_and_bruteforce]),
    "keys_normaliser_per_key_count": ("attn_importance_keys", _keys_mutant("per_key_count"),
                                      [P.test_importance_keys_match_whole_prompt,
                                       P.test_importance_keys_harmonic_and_bruteforce]),
    "head_mse_grad_sign": ("head_loss_and_grads", _head_mutant("mse_grad_sign"),
                           [lambda: P.test_head_gradients_match_finite_differences("relu")]),
    "head_no_batch_mean": ("head_loss_and_grads", _head_mutant("no_batch_mean"),
                           [lambda: P.test_head_gradients_match_finite_differences("relu")]),
    "head_w2_grad_from_z": ("head_loss_and_grads", _head_mutant("w2_grad_from_z"),
                            [lambda: P.test_head_gradients_match_finite_differences("gelu_tanh")]),
    "head_act_grad_of_output": ("head_loss_and_grads", _head_mutant("act_grad_of_output"),
                                [lambda: P.test_head_gradients_match_finite_differences("gelu_tanh")]),
    "head_hard_labels": ("head_loss_and_grads", _head_mutant("hard_labels"),
                         [P.test_head_loss_soft_labels_by_hand]),
    "adamw_no_bias_correction": ("adamw_step", _adamw_mutant("no_bias_correction"), [P.test_adamw_closed_forms]),
    "adamw_coupled_decay": ("adamw_step", _adamw_mutant("coupled_decay"), [P.test_adamw_closed_forms]),
    "adamw_eps_inside_sqrt": ("adamw_step", _adamw_mutant("eps_inside_sqrt"), [P.test_adamw_closed_forms]),
    "misalignment_ties_by_higher_index": ("misalignment_counts", _misalignment_mutant("ties_by_higher_index"),
                                          [P.test_misalignment_by_hand, P.test_misalignment_bruteforce_ranks]),
    "misalignment_ceil_counts": ("misalignment_counts", _misalignment_mutant("ceil_counts"),
                                 [P.test_misalignment_by_hand, P.test_misalignment_bruteforce_ranks]),
    "misalignment_low_high_swapped": ("misalignment_counts", _misalignment_mutant("low_high_swapped"),
                                      [P.test_misalignment_by_hand, P.test_misalignment_bruteforce_ranks]),
    "sjf_jct_uses_batch_max": ("sjf_padding", _sjf_jct_uses_max, [P.test_sjf_padding_by_hand]),
}


@pytest.mark.parametrize("name", list(LATER_MUTANTS))
def test_later_mutant_caught(name, monkeypatch):
    attr, fn, pins = LATER_MUTANTS[name]
    monkeypatch.setattr(oracle, attr, fn)
    caught = False
    for pin in pins:
        try:
            with np.errstate(all="ignore"):
                pin()
        except Exception:
            caught = True
            break
    assert caught, name


def test_later_pins_pass_unmutated():
    for _, _, pins in LATER_MUTANTS.values():
        for pin in pins:
            pin()
