"""Randomised properties of the oracle (CPU), over shapes and values drawn by hypothesis.

The pins in test_oracle_pins.py fix the oracle on hand-chosen inputs; these check identities that the
definitions imply for any input, so that a slip which happens to pass a fixed example still fails:

* Eq. 2: 0 <= H <= ln V; H is invariant under a permutation of the vocabulary; duplicating every
  vocabulary row adds exactly ln 2; a zero LM head gives ln V.  The mode is the first copy's index.
* Eq. 1: every prompt's S sums to L; packing prompts together equals scoring them apart; repeating
  each KV head over its group (GQA to MHA) changes nothing; zero queries give the harmonic form.
* Eq. 3-5: the weights of each prompt sum to 1; a shift of S or H by a constant changes nothing
  without scaling; lambda = 0 is the mean; pooling is linear in X and exact on constant rows.
* Eq. 7 / SJF: the order sorts y-hat ascending with ties by index.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from synth import inputs as I

SETTINGS = settings(max_examples=25, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def _rng(seed):
    return np.random.default_rng(seed)


@SETTINGS
@given(n=st.integers(1, 12), d=st.integers(1, 40), V=st.integers(1, 300), scale=st.floats(0.01, 8.0),
       seed=st.integers(0, 2**31 - 1))
def test_entropy_properties(n, d, V, scale, seed):
    g = _rng(seed)
    X = g.standard_normal((n, d))
    W = g.standard_normal((V, d)) * scale
    H = oracle.token_entropy(X, W)
    assert np.all(H >= -1e-12) and np.all(H <= np.log(V) + 1e-12)
    perm = g.permutation(V)
    np.testing.assert_allclose(oracle.token_entropy(X, W[perm]), H, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(oracle.token_entropy(X, np.repeat(W, 2, axis=0)), H + np.log(2), rtol=1e-10,
                               atol=1e-12)
    np.testing.assert_allclose(oracle.token_entropy(X, np.zeros_like(W)), np.log(V), rtol=1e-12)
    # the mode of the duplicated vocabulary is the first copy of the original mode
    m = oracle.vocab_argmax(X, W)
    assert np.array_equal(oracle.vocab_argmax(X, np.repeat(W, 2, axis=0)), 2 * m)
    z = X @ W.T
    assert np.array_equal(z[np.arange(n), m], z.max(axis=1))


def _qk(g, lengths, L, Hq, Hkv, dh, qscale):
    n = sum(lengths)
    Q = g.standard_normal((L, n, Hq, dh)).astype(np.float32) * qscale
    K = g.standard_normal((L, n, Hkv, dh)).astype(np.float32)
    return Q, K, I.cu_seqlens_from_lengths(lengths)


@SETTINGS
@given(lengths=st.lists(st.integers(1, 40), min_size=1, max_size=4), L=st.integers(1, 3),
       Hkv=st.sampled_from([1, 2]), G=st.sampled_from([1, 2, 3]), dh=st.sampled_from([2, 4, 8]),
       qscale=st.floats(0.1, 4.0), seed=st.integers(0, 2**31 - 1))
def test_importance_properties(lengths, L, Hkv, G, dh, qscale, seed):
    g = _rng(seed)
    Hq = Hkv * G
    Q, K, cu = _qk(g, lengths, L, Hq, Hkv, dh, qscale)
    S = oracle.attn_importance(Q, K, cu)
    assert np.all(S > 0)
    sums = np.add.reduceat(S, cu[:-1].astype(np.int64))
    np.testing.assert_allclose(sums, L, rtol=1e-10)
    # packing independence: each prompt scored alone
    for b in range(len(lengths)):
        lo, hi = int(cu[b]), int(cu[b + 1])
        alone = oracle.attn_importance(Q[:, lo:hi], K[:, lo:hi], np.array([0, hi - lo]))
        np.testing.assert_allclose(S[lo:hi], alone, rtol=1e-10)
    # GQA equals MHA with every KV head repeated over its group
    mha = oracle.attn_importance(Q, np.repeat(K, G, axis=2), cu)
    np.testing.assert_allclose(S, mha, rtol=1e-10)
    # zero queries: uniform causal rows, S_j = L (H_N - H_j) / N with harmonic numbers
    S0 = oracle.attn_importance(np.zeros_like(Q), K, cu)
    for b, N in enumerate(lengths):
        harm = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, N + 1))])
        j = np.arange(N)
        np.testing.assert_allclose(S0[cu[b]:cu[b + 1]], L * (harm[N] - harm[j]) / N, rtol=1e-10)


@SETTINGS
@given(lengths=st.lists(st.integers(1, 30), min_size=1, max_size=5), d=st.integers(1, 16),
       l1=st.floats(0.0, 2.0), l2=st.floats(0.0, 2.0), alpha=st.floats(0.2, 5.0),
       norm=st.sampled_from(["none", "zscore", "minmax"]), shift=st.floats(-5.0, 5.0),
       seed=st.integers(0, 2**31 - 1))
def test_combine_pool_properties(lengths, d, l1, l2, alpha, norm, shift, seed):
    g = _rng(seed)
    n = sum(lengths)
    S = g.random(n) * 0.1
    H = g.random(n) * 8
    cu = I.cu_seqlens_from_lengths(lengths)
    e, top = oracle.combine_weights(S, H, cu, l1, l2, alpha, norm)
    np.testing.assert_allclose(np.add.reduceat(e, cu[:-1].astype(np.int64)), 1.0, rtol=1e-12)
    for b in range(len(lengths)):
        lo, hi = int(cu[b]), int(cu[b + 1])
        assert lo <= top[b] < hi and e[top[b]] == e[lo:hi].max()
    # a constant shift of both scores changes no weight (per-prompt scaling removes it too)
    e2, _ = oracle.combine_weights(S + shift, H + shift, cu, l1, l2, alpha, norm)
    np.testing.assert_allclose(e2, e, rtol=1e-8, atol=1e-14)
    # lambda = 0: every prompt's weights are uniform
    e0, _ = oracle.combine_weights(S, H, cu, 0.0, 0.0, alpha, norm)
    np.testing.assert_allclose(e0, np.repeat(1.0 / np.array(lengths), lengths), rtol=1e-12)
    # pooling: linear in X, exact on constant rows
    X1, X2 = g.standard_normal((n, d)), g.standard_normal((n, d))
    np.testing.assert_allclose(oracle.pool(2 * X1 - 3 * X2, e, cu), 2 * oracle.pool(X1, e, cu) - 3 * oracle.pool(X2, e, cu),
                               rtol=1e-9, atol=1e-12)
    rows = g.standard_normal((len(lengths), d))
    const = np.repeat(rows, lengths, axis=0)
    np.testing.assert_allclose(oracle.pool(const, e, cu), rows, rtol=1e-10, atol=1e-12)


@SETTINGS
@given(B=st.integers(1, 40), d=st.integers(1, 12), Hd=st.integers(1, 12), K=st.integers(1, 6),
       act=st.sampled_from(["relu", "gelu_tanh"]), seed=st.integers(0, 2**31 - 1))
def test_predict_order_properties(B, d, Hd, K, act, seed):
    g = _rng(seed)
    P = g.standard_normal((B, d))
    W1, b1 = g.standard_normal((Hd, d)), g.standard_normal(Hd)
    W2, b2 = g.standard_normal((K, Hd)), g.standard_normal(K)
    c = np.sort(g.uniform(1, 100, size=K))
    y, bins, order = oracle.predict(P, W1, b1, W2, b2, c if K > 1 else None, act)
    assert sorted(order.tolist()) == list(range(B))
    ys = y[order]
    for k in range(B - 1):
        assert ys[k] < ys[k + 1] or (ys[k] == ys[k + 1] and order[k] < order[k + 1])
    if K > 1:
        # y-hat is a convex combination of the centres
        assert np.all(y >= c.min() - 1e-9) and np.all(y <= c.max() + 1e-9)
        assert np.all((bins >= 0) & (bins < K))
