"""Pins of the fp64 oracle against what the paper's definitions and mathematics fix.

Each ``pin_*`` function takes the implementation under test as an argument,
so the same checks run on the oracle (must pass) and on copies of it with a
planted mistake (``tests/test_oracle_mutants.py``: each must fail at least
one pin).  Nothing here re-types the oracle's formula: the expected values
are closed forms, invariants, special cases, library routines or a separate
pure-Python brute force.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
from oracle import bruteforce

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _ev(v):
    if isinstance(v, str):
        return float(eval(v, {"log": math.log, "Fraction": Fraction, "exp": math.exp, "sqrt": math.sqrt}))
    if isinstance(v, list):
        return [_ev(x) for x in v]
    return float(v)


def _rng(seed=0):
    return np.random.default_rng(seed)


# ============================================================================ entropy (Eq. 2)

def pin_entropy_uniform(token_entropy):
    # W = 0 or all W rows equal: every logit equal, P uniform, H = ln V exactly
    for V in (7, 1000, 151936 // 64):
        X = _rng(1).standard_normal((3, 16))
        H0 = token_entropy(X, np.zeros((V, 16)))
        np.testing.assert_allclose(H0, math.log(V), rtol=0, atol=1e-12)
        row = _rng(2).standard_normal(16)
        H1 = token_entropy(X, np.tile(row, (V, 1)))
        np.testing.assert_allclose(H1, math.log(V), rtol=0, atol=1e-11)


def pin_entropy_one_hot(token_entropy):
    # z = (a at one index, 0 elsewhere) with a = 100: H = ln(e^a + V - 1) - a e^a / (e^a + V - 1),
    # evaluated stably as log1p(c) + a c/(1+c) with c = (V-1) e^-a.  About 3.8e-39: effectively 0.
    V, a = 1000, 100.0
    X = np.zeros((1, 4)); X[0, 0] = 1.0
    W = np.zeros((V, 4)); W[17, 0] = a
    c = (V - 1) * math.exp(-a)
    expect = math.log1p(c) + a * c / (1 + c)
    H = token_entropy(X, W)[0]
    # fp64 resolves the partition sum only to ~1e-16 relative (log(1 + c) rounds to 0), so the
    # bound is absolute: the result must be 0 to within fp64 rounding of a logit of size a
    assert H >= 0.0
    assert abs(H - expect) <= 1e-13
    assert H < 1e-30


def pin_entropy_closed_form(token_entropy):
    # z = (a, 0, ..., 0): H = ln(e^a + V - 1) - a e^a / (e^a + V - 1)
    for V, a in ((10, 3.0), (1000, -2.5), (50, 0.7), (2, 5.0)):
        X = np.array([[a, 0.0]])
        W = np.zeros((V, 2)); W[0, 0] = 1.0
        expect = math.log(math.exp(a) + V - 1) - a * math.exp(a) / (math.exp(a) + V - 1)
        np.testing.assert_allclose(token_entropy(X, W)[0], expect, rtol=1e-13, atol=1e-14)


def pin_entropy_two_maxima(token_entropy):
    # two tied logits far above the rest: P -> (1/2, 1/2), H -> ln 2
    V = 500
    X = np.array([[1.0]])
    W = np.zeros((V, 1)); W[3, 0] = 80.0; W[400, 0] = 80.0
    np.testing.assert_allclose(token_entropy(X, W)[0], math.log(2), rtol=0, atol=1e-30 + 1e-12)


def pin_entropy_textbook(token_entropy):
    # logits z = ln q for a distribution q give P = q, so H is the textbook entropy of q
    q = np.array([0.5, 0.25, 0.125, 0.125])
    X = np.array([[1.0]])
    W = np.log(q)[:, None]
    np.testing.assert_allclose(token_entropy(X, W)[0], 1.75 * math.log(2), rtol=1e-14)
    # and against scipy's entropy of the softmax (a library routine the oracle does not use)
    X = _rng(3).standard_normal((5, 24))
    W = _rng(4).standard_normal((300, 24)) * 0.7
    z = X @ W.T
    ref = scipy.stats.entropy(scipy.special.softmax(z, axis=1), axis=1)
    np.testing.assert_allclose(token_entropy(X, W), ref, rtol=1e-12, atol=1e-13)


def pin_entropy_bounds_and_invariance(token_entropy):
    X = _rng(5).standard_normal((6, 12)) * 3
    W = _rng(6).standard_normal((97, 12))
    H = token_entropy(X, W)
    assert np.all(H >= 0) and np.all(H <= math.log(97) + 1e-12)
    # permuting the vocabulary does not change the entropy; rows are independent
    perm = _rng(7).permutation(97)
    np.testing.assert_allclose(token_entropy(X, W[perm]), H, rtol=1e-12)
    np.testing.assert_allclose(token_entropy(X[::-1], W), H[::-1], rtol=1e-12)


def pin_entropy_bruteforce(token_entropy):
    X = _rng(8).standard_normal((4, 6))
    W = _rng(9).standard_normal((13, 6)) * 1.5
    ref = bruteforce.entropy_rows(X.tolist(), W.tolist())
    np.testing.assert_allclose(token_entropy(X, W), ref, rtol=1e-12, atol=1e-14)


ENTROPY_PINS = [pin_entropy_uniform, pin_entropy_one_hot, pin_entropy_closed_form, pin_entropy_two_maxima,
                pin_entropy_textbook, pin_entropy_bounds_and_invariance, pin_entropy_bruteforce]


# ============================================================================ next-token mode (Eq. 2)

def pin_argmax_one_hot(vocab_argmax):
    # x = e_0 and one row k with a large first weight: the mode is k, wherever k is
    V = 300
    W = _rng(50).uniform(-1, 1, (V, 3))
    X = np.array([[1.0, 0.0, 0.0], [1.0, 0.0, 0.0]])
    for k in (0, 137, V - 1):
        Wk = W.copy(); Wk[k, 0] = 10.0
        assert list(vocab_argmax(X, Wk)) == [k, k]


def pin_argmax_ties_lowest(vocab_argmax):
    # equal largest logits: the lowest vocabulary index wins (also the worked example in tests/golden)
    V = 500
    W = _rng(51).uniform(-1, 1, (V, 2)); W[[3, 77, 400], 0] = 50.0; W[[3, 77, 400], 1] = 0.0
    assert list(vocab_argmax(np.array([[1.0, 0.25]]), W)) == [3]
    for ex in _golden()["vocab_argmax"]:
        assert list(vocab_argmax(np.array(ex["X"]), np.array(ex["W"]))) == ex["argmax"]


def pin_argmax_permutation(vocab_argmax):
    # permuting the vocabulary rows moves the mode with them (continuous random logits: no ties)
    X = _rng(52).standard_normal((9, 16)); W = _rng(53).standard_normal((211, 16))
    a = vocab_argmax(X, W)
    perm = _rng(54).permutation(211)
    b = vocab_argmax(X, W[perm])
    np.testing.assert_array_equal(perm[b], a)


def pin_argmax_bruteforce(vocab_argmax):
    # scalar loops: exact logits by fsum, first strict maximum; and the mode of scipy's softmax
    X = _rng(55).standard_normal((5, 6)); W = _rng(56).standard_normal((40, 6))
    got = vocab_argmax(X, W)
    for i in range(5):
        z = [math.fsum(W[v, k] * X[i, k] for k in range(6)) for v in range(40)]
        best = 0
        for v in range(1, 40):
            if z[v] > z[best]:
                best = v
        assert got[i] == best
        assert got[i] == int(np.argmax(scipy.special.softmax(np.array(z))))


ARGMAX_PINS = [pin_argmax_one_hot, pin_argmax_ties_lowest, pin_argmax_permutation, pin_argmax_bruteforce]


# ============================================================================ importance (Eq. 1)

def _harm(n):
    return math.fsum(1.0 / k for k in range(1, n + 1))


def pin_importance_row_stochastic(attn_importance):
    # every causal softmax row sums to 1, so sum_j S_j = (1/N) * N = 1 per layer and prompt
    L, Hq, Hkv, dh = 3, 4, 2, 8
    lengths = [5, 1, 17]
    n = sum(lengths)
    Q = _rng(10).standard_normal((L, n, Hq, dh)) * 2
    K = _rng(11).standard_normal((L, n, Hkv, dh))
    cu = np.concatenate([[0], np.cumsum(lengths)])
    S = attn_importance(Q, K, cu)
    assert np.all(S > 0)
    for b in range(len(lengths)):
        np.testing.assert_allclose(S[cu[b]:cu[b + 1]].sum(), L, rtol=1e-13)


def pin_importance_uniform_harmonic(attn_importance):
    # Q = 0: every row uniform over j <= i, A_ij = 1/(i+1); column j collects H_N - H_j
    N, L = 37, 2
    Q = np.zeros((L, N, 4, 8))
    K = _rng(12).standard_normal((L, N, 1, 8))
    S = attn_importance(Q, K, [0, N])
    expect = [L * (_harm(N) - _harm(j)) / N for j in range(N)]
    np.testing.assert_allclose(S, expect, rtol=1e-13)


def pin_importance_edges(attn_importance):
    # query 0 sees only key 0 (A_00 = 1); the last key receives only the last query's own mass;
    # a one-token prompt has S = L
    N, Hq, dh = 9, 3, 4
    Q = _rng(13).standard_normal((1, N, Hq, dh)) * 2
    K = _rng(14).standard_normal((1, N, Hq, dh))
    S = attn_importance(Q, K, [0, N], scale=0.8)
    last = 0.0
    for h in range(Hq):
        s = 0.8 * Q[0, N - 1, h] @ K[0, :, h].T
        last += math.exp(s[-1]) / math.fsum(np.exp(s)) / Hq
    np.testing.assert_allclose(S[N - 1], last / N, rtol=1e-13)
    S1 = attn_importance(Q[:, :1], K[:, :1], [0, 1])
    np.testing.assert_allclose(S1, [1.0], rtol=1e-15)
    # two tokens, one head: A_10 = 1 / (1 + exp(s_11 - s_10)); S = ((1 + A_10)/2, (1 - A_10)/2)
    q = np.array([[[[0.3]], [[1.7]]]]); k = np.array([[[[-0.4]], [[0.9]]]])
    a10 = 1.0 / (1.0 + math.exp(1.7 * 0.9 - 1.7 * -0.4))
    np.testing.assert_allclose(attn_importance(q, k, [0, 2], scale=1.0), [(1 + a10) / 2, (1 - a10) / 2], rtol=1e-14)


def pin_importance_gqa(attn_importance):
    # grouped-query attention equals multi-head attention with each key head repeated G times
    L, N, Hq, Hkv, dh = 2, 11, 6, 2, 4
    Q = _rng(15).standard_normal((L, N, Hq, dh))
    K = _rng(16).standard_normal((L, N, Hkv, dh))
    Krep = np.repeat(K, Hq // Hkv, axis=2)
    np.testing.assert_allclose(attn_importance(Q, K, [0, N]), attn_importance(Q, Krep, [0, N]), rtol=1e-13)


def pin_importance_packing(attn_importance):
    # a packed batch equals its prompts run separately; order of prompts only permutes the output
    lengths = [4, 9, 2]
    n = sum(lengths)
    Q = _rng(17).standard_normal((1, n, 2, 4))
    K = _rng(18).standard_normal((1, n, 2, 4))
    cu = np.concatenate([[0], np.cumsum(lengths)])
    S = attn_importance(Q, K, cu)
    for b in range(3):
        lo, hi = cu[b], cu[b + 1]
        np.testing.assert_allclose(S[lo:hi], attn_importance(Q[:, lo:hi], K[:, lo:hi], [0, hi - lo]), rtol=1e-13)


def pin_importance_bruteforce(attn_importance):
    lengths = [5, 3]
    n = sum(lengths)
    Q = _rng(19).standard_normal((n, 4, 3))
    K = _rng(20).standard_normal((n, 2, 3))
    S = attn_importance(Q[None], K[None], np.concatenate([[0], np.cumsum(lengths)]), scale=0.7)
    ref = bruteforce.importance(Q.tolist(), K.tolist(), lengths, 0.7)
    np.testing.assert_allclose(S, ref, rtol=1e-12)


IMPORTANCE_PINS = [pin_importance_row_stochastic, pin_importance_uniform_harmonic, pin_importance_edges,
                   pin_importance_gqa, pin_importance_packing, pin_importance_bruteforce]


# ============================================================================ combine (Eq. 3, 4)

def pin_combine_simplex_and_average(combine_weights):
    lengths = [6, 1, 4]
    cu = np.concatenate([[0], np.cumsum(lengths)])
    S = _rng(21).random(11); H = _rng(22).random(11) * 5
    e, top = combine_weights(S, H, cu, 0.7, 0.3, 0.5)
    for b in range(3):
        np.testing.assert_allclose(e[cu[b]:cu[b + 1]].sum(), 1.0, rtol=1e-14)
    assert np.all(e > 0)
    # lambda1 = lambda2 = 0 is average pooling (ablation row "Average Pooling", Table 4)
    e0, _ = combine_weights(S, H, cu, 0.0, 0.0, 1.0)
    np.testing.assert_allclose(e0, np.repeat([1 / 6, 1.0, 1 / 4], lengths), rtol=1e-14)


def pin_combine_two_token_logistic(combine_weights):
    # N = 2: e_0 = 1 / (1 + exp((T_1 - T_0)/alpha)) with T = l1 S + l2 H
    S = np.array([0.2, 0.9]); H = np.array([3.0, 1.0])
    for l1, l2, a in ((0.4, 0.6, 1.0), (1.0, 0.0, 0.5), (0.0, 1.0, 2.0), (0.9, 0.1, 0.25)):
        T0, T1 = l1 * 0.2 + l2 * 3.0, l1 * 0.9 + l2 * 1.0
        e0 = 1.0 / (1.0 + math.exp((T1 - T0) / a))
        e, top = combine_weights(S, H, [0, 2], l1, l2, a)
        np.testing.assert_allclose(e, [e0, 1 - e0], rtol=1e-14)
        assert top[0] == (0 if e0 >= 0.5 else 1)


def pin_combine_invariances(combine_weights):
    S = _rng(23).random(9); H = _rng(24).random(9) * 4
    e, _ = combine_weights(S, H, [0, 9], 0.5, 0.5, 1.0)
    # shifting all scores of a prompt by a constant does not change e
    e2, _ = combine_weights(S + 3.0, H - 1.0, [0, 9], 0.5, 0.5, 1.0)
    np.testing.assert_allclose(e2, e, rtol=1e-13)
    # (lambda1, lambda2, alpha) -> c * (...) leaves T/alpha unchanged
    e3, _ = combine_weights(S, H, [0, 9], 1.5, 1.5, 3.0)
    np.testing.assert_allclose(e3, e, rtol=1e-13)
    # alpha -> 0 concentrates all weight on the argmax of T; large alpha -> uniform
    T = 0.5 * S + 0.5 * H
    e4, top = combine_weights(S, H, [0, 9], 0.5, 0.5, 1e-4)
    assert top[0] == int(np.argmax(T)) and e4[top[0]] > 1 - 1e-12
    e5, _ = combine_weights(S, H, [0, 9], 0.5, 0.5, 1e9)
    np.testing.assert_allclose(e5, 1 / 9, rtol=1e-8)
    # monotone: a larger fused score never gets a smaller weight
    order = np.argsort(T)
    assert np.all(np.diff(e[order]) >= 0)


def pin_combine_zscore(combine_weights):
    # with z-scoring, an affine change of S or H (positive slope a) leaves e unchanged up to the
    # epsilon in the denominator, which moves by a factor 1/a: relative effect ~ 1e-6 / (a * std)
    S = _rng(25).random(14); H = _rng(26).random(14)
    e, _ = combine_weights(S, H, [0, 14], 0.6, 0.4, 0.7, norm="zscore")
    e2, _ = combine_weights(10 * S + 4, 4 * H - 2, [0, 14], 0.6, 0.4, 0.7, norm="zscore")
    np.testing.assert_allclose(e2, e, rtol=2e-5)
    # a constant S contributes nothing after z-scoring (0 / (0 + eps))
    e3, _ = combine_weights(np.full(14, 0.3), H, [0, 14], 5.0, 0.4, 0.7, norm="zscore")
    e4, _ = combine_weights(np.full(14, 0.3), H, [0, 14], 0.0, 0.4, 0.7, norm="zscore")
    np.testing.assert_allclose(e3, e4, rtol=1e-12)


def pin_combine_zscore_by_hand(combine_weights):
    # hand-derived z-scored examples (tests/golden): population std, epsilon added to the std.
    # Sample std (ddof 1) or epsilon inside the square root change these values by 1e-2 to 1e-1.
    for ex in _golden()["combine_zscore"]:
        cu = np.concatenate([[0], np.cumsum(ex["lengths"])])
        e, top = combine_weights(np.array(ex["S"]), np.array(ex["H"]), cu, ex["lambda1"], ex["lambda2"],
                                 ex["alpha"], norm="zscore")
        u = np.array(_ev(ex["u"]))
        np.testing.assert_allclose(e, np.exp(u) / np.exp(u).sum(), rtol=1e-12)
        assert list(top) == ex["top"]


def pin_combine_bruteforce(combine_weights):
    lengths = [3, 5]
    S = _rng(27).random(8); H = _rng(28).random(8) * 2
    e, _ = combine_weights(S, H, [0, 3, 8], 0.8, 0.2, 0.6)
    np.testing.assert_allclose(e, bruteforce.fused_weights(S.tolist(), H.tolist(), lengths, 0.8, 0.2, 0.6), rtol=1e-13)


COMBINE_PINS = [pin_combine_simplex_and_average, pin_combine_two_token_logistic, pin_combine_invariances,
                pin_combine_zscore, pin_combine_zscore_by_hand, pin_combine_bruteforce]


# ============================================================================ pooling (Eq. 5)

def pin_pool_mean_identity_linear(pool):
    lengths = [4, 2]
    cu = [0, 4, 6]
    X = _rng(29).standard_normal((6, 5))
    u = np.repeat([1 / 4, 1 / 2], lengths)
    np.testing.assert_allclose(pool(X, u, cu), [X[:4].mean(0), X[4:].mean(0)], rtol=1e-14)
    # identical rows pool to that row for any simplex weights
    Xs = np.tile(X[0], (6, 1))
    w = _rng(30).random(6); w[:4] /= w[:4].sum(); w[4:] /= w[4:].sum()
    np.testing.assert_allclose(pool(Xs, w, cu), [X[0], X[0]], rtol=1e-14)
    # one-hot weights select the row; linear in X
    oh = np.array([0, 0, 1.0, 0, 1.0, 0])
    np.testing.assert_allclose(pool(X, oh, cu), [X[2], X[4]], rtol=0)
    Y = _rng(31).standard_normal((6, 5))
    np.testing.assert_allclose(pool(2 * X - Y, w, cu), 2 * pool(X, w, cu) - pool(Y, w, cu), rtol=1e-12, atol=1e-14)


def pin_pool_bruteforce(pool):
    X = _rng(32).standard_normal((7, 3)); e = _rng(33).random(7)
    np.testing.assert_allclose(pool(X, e, [0, 2, 7]), bruteforce.pooled(X.tolist(), e.tolist(), [2, 5]), rtol=1e-13)


POOL_PINS = [pin_pool_mean_identity_linear, pin_pool_bruteforce]


# ============================================================================ length head (Eq. 7)

def pin_predict_mlp(predict):
    # K = 1 is a plain 2-layer MLP: checked against explicit scalar loops
    B, d, Hd = 3, 5, 4
    h = _rng(34).standard_normal((B, d)); W1 = _rng(35).standard_normal((Hd, d)); b1 = _rng(36).standard_normal(Hd)
    W2 = _rng(37).standard_normal((1, Hd)); b2 = np.array([0.25])
    y, bins, order = predict(h, W1, b1, W2, b2, None, "relu")
    for i in range(B):
        a = [max(0.0, math.fsum(W1[j, k] * h[i, k] for k in range(d)) + b1[j]) for j in range(Hd)]
        o = math.fsum(W2[0, j] * a[j] for j in range(Hd)) + 0.25
        assert abs(y[i] - o) < 1e-12
    assert bins is None
    assert list(order) == sorted(range(B), key=lambda i: (y[i], i))


def pin_predict_bins(predict):
    # W2 = 0, b2 = 0: uniform p-hat, y-hat is the mean of the centres
    h = _rng(38).standard_normal((4, 3)); W1 = _rng(39).standard_normal((6, 3))
    c = np.array([10.0, 50.0, 90.0, 400.0, 1000.0])
    y, bins, _ = predict(h, W1, None, np.zeros((5, 6)), np.zeros(5), c, "relu")
    np.testing.assert_allclose(y, c.mean(), rtol=1e-14)
    assert list(bins) == [0, 0, 0, 0]
    # one dominant logit: y-hat = c_k, bin = k
    b2 = np.zeros(5); b2[3] = 200.0
    y, bins, _ = predict(h, W1, None, np.zeros((5, 6)), b2, c, "relu")
    np.testing.assert_allclose(y, 400.0, rtol=1e-12)
    assert list(bins) == [3] * 4


def pin_predict_order_stable(predict):
    # ties in y-hat keep prompt order (shortest job first, Section 5.4)
    h = np.array([[1.0], [0.0], [1.0], [-1.0], [0.0]])
    y, _, order = predict(h, np.eye(1), None, np.eye(1), None, None, "relu")
    np.testing.assert_allclose(y, [1, 0, 1, 0, 0])
    assert list(order) == [1, 3, 4, 0, 2]


def pin_predict_gelu(predict):
    # tanh-GELU: 0 at 0, close to the exact GELU x * Phi(x), close to x for large x
    xs = np.array([[-3.0], [-0.5], [0.0], [0.7], [6.0]])
    y, _, _ = predict(xs, np.eye(1), None, np.eye(1), None, None, "gelu_tanh")
    exact = [x * 0.5 * (1 + math.erf(x / math.sqrt(2))) for x in xs[:, 0]]
    np.testing.assert_allclose(y, exact, atol=2e-3)
    assert y[2] == 0.0 and abs(y[4] - 6.0) < 1e-6


def pin_predict_gelu_tanh_values(predict):
    # the tanh form of GELU at worked points (tests/golden) and against PyTorch's own
    # gelu(approximate="tanh") in fp64 on a grid; the exact erf form misses by 1e-5 to 4e-4
    import torch
    ex = _golden()["predict_gelu_tanh"][0]
    xs = np.array(ex["x"])[:, None]
    y, _, _ = predict(xs, np.eye(1), None, np.eye(1), None, None, "gelu_tanh")
    np.testing.assert_allclose(y, ex["yhat"], rtol=1e-12, atol=1e-15)
    grid = np.linspace(-6.0, 6.0, 97)[:, None]
    y, _, _ = predict(grid, np.eye(1), None, np.eye(1), None, None, "gelu_tanh")
    ref = torch.nn.functional.gelu(torch.from_numpy(grid[:, 0].copy()), approximate="tanh").numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-15)


PREDICT_PINS = [pin_predict_mlp, pin_predict_bins, pin_predict_order_stable, pin_predict_gelu,
                pin_predict_gelu_tanh_values]


# ============================================================================ runs on the oracle

@pytest.mark.parametrize("pin", ENTROPY_PINS, ids=lambda f: f.__name__)
def test_entropy_pins(pin):
    pin(oracle.token_entropy)


@pytest.mark.parametrize("pin", ARGMAX_PINS, ids=lambda f: f.__name__)
def test_argmax_pins(pin):
    pin(oracle.vocab_argmax)


@pytest.mark.parametrize("pin", IMPORTANCE_PINS, ids=lambda f: f.__name__)
def test_importance_pins(pin):
    pin(oracle.attn_importance)


@pytest.mark.parametrize("pin", COMBINE_PINS, ids=lambda f: f.__name__)
def test_combine_pins(pin):
    pin(oracle.combine_weights)


@pytest.mark.parametrize("pin", POOL_PINS, ids=lambda f: f.__name__)
def test_pool_pins(pin):
    pin(oracle.pool)


@pytest.mark.parametrize("pin", PREDICT_PINS, ids=lambda f: f.__name__)
def test_predict_pins(pin):
    pin(oracle.predict)


def test_importance_row_chunks_complete():
    # splitting the query rows into chunks only splits the column sum
    Q = _rng(40).standard_normal((1, 23, 2, 4)); K = _rng(41).standard_normal((1, 23, 2, 4))
    np.testing.assert_allclose(oracle.attn_importance(Q, K, [0, 23], row_chunk=5),
                               oracle.attn_importance(Q, K, [0, 23], row_chunk=4096), rtol=1e-14)


def test_importance_tail_matches_whole_prompt():
    # the last m keys only receive attention from the last m queries: the tail form is exact
    N, L = 53, 2
    Q = _rng(42).standard_normal((L, N, 4, 8)) * 1.5
    K = _rng(43).standard_normal((L, N, 2, 8))
    full = oracle.attn_importance(Q, K, [0, N])
    for m in (1, 7, N):
        np.testing.assert_allclose(oracle.attn_importance_tail(Q, K, N, m), full[N - m:], rtol=1e-13)
    # and on the uniform case, the harmonic closed form
    Q0 = np.zeros((1, N, 2, 4))
    tail = oracle.attn_importance_tail(Q0, K[:1, :, :2, :4], N, 10)
    np.testing.assert_allclose(tail, [(_harm(N) - _harm(j)) / N for j in range(N - 10, N)], rtol=1e-13)


def test_importance_keys_match_whole_prompt():
    # any key set of one prompt, from the rows that reach it: equal to the whole-prompt S there,
    # to the tail form on the last keys, and the head partition sums to the full head average
    N, L = 61, 2
    Q = _rng(44).standard_normal((L, N, 4, 8)) * 1.5
    K = _rng(45).standard_normal((L, N, 2, 8))
    full = oracle.attn_importance(Q, K, [0, N])
    for keys, chunk in (([0], 256), ([0, 1, 2, 30, 60], 7), (list(range(20, 45)), 5), ([60, 5, 33], 13)):
        np.testing.assert_allclose(oracle.attn_importance_keys(Q, K, N, keys, row_chunk=chunk), full[keys],
                                   rtol=1e-13)
    np.testing.assert_allclose(oracle.attn_importance_keys(Q, K, N, range(N - 9, N)),
                               oracle.attn_importance_tail(Q, K, N, 9), rtol=1e-13)
    parts = sum(oracle.attn_importance_keys(Q, K, N, [0, 17], heads=[h]) for h in range(4))
    np.testing.assert_allclose(parts, full[[0, 17]], rtol=1e-13)


def test_importance_keys_harmonic_and_bruteforce():
    # Q = 0: uniform causal rows, S_j = (H_N - H_j) / N on any key set; and the pure-Python brute force
    N = 40
    K = _rng(46).standard_normal((1, N, 1, 4))
    got = oracle.attn_importance_keys(np.zeros((1, N, 2, 4)), K, N, [0, 7, 39], row_chunk=6)
    np.testing.assert_allclose(got, [(_harm(N) - _harm(j)) / N for j in (0, 7, 39)], rtol=1e-13)
    n = 7
    Q = _rng(47).standard_normal((n, 2, 3)); Kb = _rng(48).standard_normal((n, 1, 3))
    ref = bruteforce.importance(Q.tolist(), Kb.tolist(), [n], 0.6)
    got = oracle.attn_importance_keys(Q, Kb, n, [1, 4, 6], scale=0.6, row_chunk=2)
    np.testing.assert_allclose(got, [ref[1], ref[4], ref[6]], rtol=1e-13)


def test_widen_bf16_exact():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0001, 0x7F7F, 0x0000], dtype=np.uint16)
    got = oracle.widen(bits)
    assert got[0] == 1.0 and got[1] == -1.0 and got[5] == 0.0
    assert got[2] == 3.140625
    assert got[3] == 2.0 ** -133
    assert got[4] == (2 - 2 ** -7) * 2.0 ** 127


# ============================================================================ golden worked examples

def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_golden_entropy():
    for ex in _golden()["entropy"]:
        H = oracle.token_entropy(np.array(_ev(ex["X"])), np.array(_ev(ex["W"])))
        np.testing.assert_allclose(H, _ev(ex["H"]), rtol=1e-14, atol=1e-15)


def test_golden_importance():
    for ex in _golden()["importance"]:
        Q = np.array(_ev(ex["Q"]))[None]; K = np.array(_ev(ex["K"]))[None]
        cu = np.concatenate([[0], np.cumsum(ex["lengths"])])
        S = oracle.attn_importance(Q, K, cu, scale=ex["scale"])
        np.testing.assert_allclose(S, _ev(ex["S"]), rtol=1e-14)


def test_golden_combine_pool():
    for ex in _golden()["combine_pool"]:
        cu = np.concatenate([[0], np.cumsum(ex["lengths"])])
        e, top = oracle.combine_weights(np.array(_ev(ex["S"])), np.array(_ev(ex["H"])), cu,
                                        ex["lambda1"], ex["lambda2"], ex["alpha"])
        np.testing.assert_allclose(e, _ev(ex["e"]), rtol=1e-14)
        assert list(top) == ex["top"]
        np.testing.assert_allclose(oracle.pool(np.array(_ev(ex["X"])), e, cu), _ev(ex["pooled"]), rtol=1e-14)


def test_golden_predict():
    for ex in _golden()["predict"]:
        y, bins, order = oracle.predict(np.array(_ev(ex["pooled"])), np.array(_ev(ex["W1"])), np.array(_ev(ex["b1"])),
                                        np.array(_ev(ex["W2"])), np.array(_ev(ex["b2"])), np.array(ex["centres"]))
        np.testing.assert_allclose(y, _ev(ex["yhat"]), rtol=1e-14)
        assert list(bins) == ex["bin"]


# ============================================================================ Eq. 6 and Eq. 8

def test_soft_labels():
    for K, i in ((5, 0), (9, 4), (12, 11)):
        p = oracle.soft_labels(i, K)
        np.testing.assert_allclose(p.sum(), 1.0, rtol=1e-15)
        assert int(np.argmax(p)) == i
        # neighbours decay by exactly e^-1 per bin
        for j in range(K - 1):
            if j >= i:
                np.testing.assert_allclose(p[j + 1] / p[j], math.exp(-1), rtol=1e-14)
        # symmetric about the true bin
        for t in range(1, K):
            if 0 <= i - t and i + t < K:
                np.testing.assert_allclose(p[i - t], p[i + t], rtol=1e-15)


def test_length_loss():
    p = np.array([[0.2, 0.8]]); phat = np.array([[0.5, 0.5]])
    # lambda3 = 1: pure cross-entropy = ln 2; lambda3 = 0: pure MSE
    np.testing.assert_allclose(oracle.length_loss(p, phat, [3.0], [1.0], 1.0), math.log(2), rtol=1e-15)
    np.testing.assert_allclose(oracle.length_loss(p, phat, [3.0], [1.0], 0.0), 4.0, rtol=1e-15)
    # CE(p, p) is the entropy of p (Gibbs): minimum over p-hat
    ce_pp = oracle.length_loss(p, p, [0.0], [0.0], 1.0)
    np.testing.assert_allclose(ce_pp, scipy.stats.entropy(p[0]), rtol=1e-14)
    assert oracle.length_loss(p, phat, [0.0], [0.0], 1.0) > ce_pp


# ============================================================================ row normalisers (prefill LSE)

def test_row_lse_bruteforce():
    # two prompts, grouped heads: every row's log partition sum against scalar loops
    lengths = [5, 3]
    Q = _rng(50).standard_normal((1, 8, 4, 3)) * 1.3
    K = _rng(51).standard_normal((1, 8, 2, 3))
    got = oracle.attn_row_lse(Q, K, [0, 5, 8], scale=0.7)
    ref = bruteforce.row_lse(Q[0].tolist(), K[0].tolist(), lengths, 0.7)
    np.testing.assert_allclose(got[0], np.array(ref), rtol=1e-13, atol=1e-13)


def test_row_lse_closed_forms():
    # the first row of a prompt sees only itself: lse = scale q.k; zero queries: lse_i = log(i + 1)
    Q = _rng(52).standard_normal((2, 9, 2, 4)); K = _rng(53).standard_normal((2, 9, 1, 4))
    lse = oracle.attn_row_lse(Q, K, [0, 4, 9], scale=0.5)
    for l in range(2):
        for h in range(2):
            for lo in (0, 4):
                assert lse[l, h, lo] == pytest.approx(0.5 * Q[l, lo, h] @ K[l, lo, 0], rel=1e-14)
    z = oracle.attn_row_lse(np.zeros((1, 6, 2, 4)), K[:1, :6], [0, 6])
    np.testing.assert_allclose(z[0, 1], np.log(np.arange(1, 7)), rtol=1e-14)


def test_importance_from_lse_bruteforce_and_identity():
    lengths = [6, 2]
    Q = _rng(54).standard_normal((1, 8, 2, 3)) * 1.2
    K = _rng(55).standard_normal((1, 8, 1, 3))
    cu = [0, 6, 8]
    # with the exact normalisers the rows are softmax rows: the plain importance
    exact = oracle.attn_row_lse(Q, K, cu, scale=0.9)
    np.testing.assert_allclose(oracle.attn_importance_from_lse(Q, K, cu, exact, scale=0.9),
                               oracle.attn_importance(Q, K, cu, scale=0.9), rtol=1e-13)
    # shifted normalisers scale row i by exp(-delta_i): scalar loops agree
    shifted = exact + _rng(56).standard_normal(exact.shape) * 0.3
    got = oracle.attn_importance_from_lse(Q, K, cu, shifted, scale=0.9)
    ref = bruteforce.importance_with_lse(Q[0].tolist(), K[0].tolist(), lengths, 0.9, shifted[0].tolist())
    np.testing.assert_allclose(got, ref, rtol=1e-13)
    # mass: sum_j S_j = (1/N) sum_i (1/Hq) sum_h exp(-delta_hi) per prompt
    delta = shifted - exact
    for lo, hi in ((0, 6), (6, 8)):
        mass = np.exp(-delta[0, :, lo:hi]).mean(axis=0).sum() / (hi - lo)
        assert got[lo:hi].sum() == pytest.approx(mass, rel=1e-13)


# ============================================================================ training the length head

def _head_problem(seed, B=5, d=6, Hd=4, K=5, act="relu"):
    g = _rng(seed)
    h = g.standard_normal((B, d))
    params = {"W1": g.standard_normal((Hd, d)) * 0.7, "b1": g.standard_normal(Hd) * 0.3,
              "W2": g.standard_normal((K, Hd)) * 0.7, "b2": g.standard_normal(K) * 0.3}
    edges = np.linspace(0.0, 50.0 * K, K + 1)
    centres = 0.5 * (edges[1:] + edges[:-1])
    y = g.uniform(-10.0, 50.0 * K + 10.0, size=B)
    return h, y, edges, centres, params


@pytest.mark.parametrize("act", ["relu", "gelu_tanh"])
def test_head_gradients_match_finite_differences(act):
    # central differences of the Eq. 8 loss pin every analytic gradient entry
    h, y, edges, centres, P = _head_problem(60, act=act)
    lam = 0.3
    # keep ReLU pre-activations away from the kink so the difference quotient is smooth
    z = h @ P["W1"].T + P["b1"]
    assert np.abs(z).min() > 1e-3
    loss, g = oracle.head_loss_and_grads(h, y, edges, centres, P["W1"], P["b1"], P["W2"], P["b2"], lam, act)
    eps = 1e-6
    for name in ("W1", "b1", "W2", "b2"):
        fd = np.zeros_like(P[name])
        for idx in np.ndindex(P[name].shape):
            Pp = {k: v.copy() for k, v in P.items()}
            Pm = {k: v.copy() for k, v in P.items()}
            Pp[name][idx] += eps
            Pm[name][idx] -= eps
            lp, _ = oracle.head_loss_and_grads(h, y, edges, centres, Pp["W1"], Pp["b1"], Pp["W2"], Pp["b2"], lam, act)
            lm, _ = oracle.head_loss_and_grads(h, y, edges, centres, Pm["W1"], Pm["b1"], Pm["W2"], Pm["b2"], lam, act)
            fd[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(g[name], fd, rtol=1e-5, atol=1e-7 * max(1.0, abs(loss)))


def test_head_loss_closed_form():
    # W2 = 0, b2 = 0: p-hat uniform over 2 bins, CE = log 2 whatever the soft labels, y-hat the mean centre
    h = np.ones((3, 4))
    W1 = np.ones((2, 4)); b1 = np.zeros(2)
    y = np.array([3.0, 15.0, 40.0])
    edges = np.array([0.0, 10.0, 20.0]); centres = np.array([5.0, 15.0])
    lam = 0.25
    loss, _ = oracle.head_loss_and_grads(h, y, edges, centres, W1, b1, np.zeros((2, 2)), np.zeros(2), lam)
    assert loss == pytest.approx(lam * math.log(2.0) + (1 - lam) * np.mean((y - 10.0) ** 2), rel=1e-14)


def test_length_bin_edges():
    edges = [0.0, 10.0, 20.0, 30.0]
    assert list(oracle.length_bin([-5.0, 0.0, 9.99, 10.0, 19.0, 20.0, 29.9, 30.0, 100.0], edges)) == \
        [0, 0, 0, 1, 1, 2, 2, 2, 2]


def test_adamw_closed_forms():
    # first step: m_hat = g, v_hat = g^2, so each coordinate moves by lr g / (|g| + eps) after decay
    th = np.array([1.0, -2.0, 0.5]); g = np.array([0.3, -4.0, 0.0])
    new, m, v = oracle.adamw_step(th, g, np.zeros(3), np.zeros(3), 1, 0.1, 0.9, 0.999, 1e-8, 0.01)
    np.testing.assert_allclose(new, th * (1 - 0.001) - 0.1 * g / (np.abs(g) + 1e-8), rtol=1e-15)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-15)
    # second step on a scalar, by hand
    m2 = 0.9 * 0.03 + 0.1 * 0.5
    v2 = 0.999 * 0.001 * 0.09 + 0.001 * 0.25
    exp = (1.0 * (1 - 0.001) - 0.1 * 0.3 / (0.3 + 1e-8)) * (1 - 0.001) \
        - 0.1 * (m2 / (1 - 0.81)) / (math.sqrt(v2 / (1 - 0.999 ** 2)) + 1e-8)
    n1, m1, v1 = oracle.adamw_step(np.array([1.0]), np.array([0.3]), np.zeros(1), np.zeros(1), 1, 0.1, 0.9, 0.999,
                                   1e-8, 0.01)
    n2, _, _ = oracle.adamw_step(n1, np.array([0.5]), m1, v1, 2, 0.1, 0.9, 0.999, 1e-8, 0.01)
    assert n2[0] == pytest.approx(exp, rel=1e-14)


def test_head_training_reduces_loss():
    # a few AdamW steps on a fixed batch lower the Eq. 8 loss
    h, y, edges, centres, P = _head_problem(61, B=16, d=8, Hd=16, K=6)
    M = {k: np.zeros_like(v) for k, v in P.items()}
    Vv = {k: np.zeros_like(v) for k, v in P.items()}
    losses = []
    for t in range(1, 41):
        loss, _, P, M, Vv = oracle.head_train_step(h, y, edges, centres, P, M, Vv, t, 0.5, 3e-2)
        losses.append(loss)
    assert losses[-1] < 0.5 * losses[0]


# ============================================================================ importance variants

def test_importance_exclude_self_bruteforce_and_diagonal():
    lengths = [7, 4]
    Q = _rng(70).standard_normal((1, 11, 4, 3)) * 1.4
    K = _rng(71).standard_normal((1, 11, 2, 3))
    cu = [0, 7, 11]
    ex = oracle.attn_importance(Q, K, cu, scale=0.8, exclude_self=True)
    ref = bruteforce.importance(Q[0].tolist(), K[0].tolist(), lengths, 0.8, exclude_self=True)
    np.testing.assert_allclose(ex, ref, rtol=1e-13)
    # the excluded mass is the head-averaged diagonal: the first token of a prompt loses 1/N exactly
    inc = oracle.attn_importance(Q, K, cu, scale=0.8)
    assert inc[0] - ex[0] == pytest.approx(1.0 / 7, rel=1e-13)
    assert inc[7] - ex[7] == pytest.approx(1.0 / 4, rel=1e-13)
    # and through given row normalisers the same
    lse = oracle.attn_row_lse(Q, K, cu, scale=0.8)
    np.testing.assert_allclose(oracle.attn_importance_from_lse(Q, K, cu, lse, scale=0.8, exclude_self=True), ex,
                               rtol=1e-13)


def test_importance_layer_weights_linear():
    Q = _rng(72).standard_normal((3, 9, 2, 4)); K = _rng(73).standard_normal((3, 9, 1, 4))
    cu = [0, 5, 9]
    w = [0.5, -1.0, 2.0]
    per_layer = [oracle.attn_importance(Q[l:l + 1], K[l:l + 1], cu) for l in range(3)]
    np.testing.assert_allclose(oracle.attn_importance(Q, K, cu, layer_weights=w),
                               sum(wl * s for wl, s in zip(w, per_layer)), rtol=1e-13)


def test_combine_minmax_closed_forms():
    # min-max scaling maps each prompt's S and H onto [0, 1) affinely: weights follow by hand
    S = np.array([2.0, 4.0, 3.0, 7.0, 7.0])
    H = np.array([1.0, 0.0, 5.0, 2.0, 2.0])
    cu = [0, 3, 5]
    e, top = oracle.combine_weights(S, H, cu, 0.6, 0.4, 0.5, "minmax")
    s0 = (S[:3] - 2.0) / (2.0 + 1e-6)
    h0 = (H[:3] - 0.0) / (5.0 + 1e-6)
    u = (0.6 * s0 + 0.4 * h0) / 0.5
    np.testing.assert_allclose(e[:3], np.exp(u) / np.exp(u).sum(), rtol=1e-13)
    # a constant prompt (zero range) scales to zeros: uniform weights, first index on top
    np.testing.assert_allclose(e[3:], [0.5, 0.5], rtol=1e-15)
    assert top[1] == 3


# ============================================================================ analyses

def test_misalignment_by_hand():
    # N = 10, 40% -> 4 tokens in each of the high and low sets; ranks read off directly
    H = np.array([9, 8, 7, 6, 5, 4, 3, 2, 1, 0], dtype=float)      # high H: tokens 0-3, low H: 6-9
    S = np.array([0, 1, 9, 8, 5, 5, 7, 2, 3, 4], dtype=float)      # low S: 0, 1, 7, 8; high S: 2, 3, 6, 5
    c = oracle.misalignment_counts(H, S, [0, 10])
    # the tied 5s rank 4 before 5, so token 5 is in the top four of S and token 4 is not
    # high-H {0,1,2,3} & low-S {0,1,7,8} = {0,1}; low-H {6,7,8,9} & high-S {2,3,5,6} = {6}
    assert c.tolist() == [[4, 2, 4, 1]]
    # ties go by index: equal values, the lower index ranks lower
    c = oracle.misalignment_counts(np.zeros(5), np.arange(5.0), [0, 5], 0.4, 0.4)
    # H all equal: low-H = tokens 0,1 (lowest indices), high-H = tokens 3,4; S low = 0,1, high = 3,4
    assert c.tolist() == [[2, 0, 2, 0]]


def test_misalignment_bruteforce_ranks():
    g = _rng(80)
    H = g.integers(0, 5, size=23).astype(float)   # many ties
    S = g.standard_normal(23)
    cu = [0, 9, 23]
    got = oracle.misalignment_counts(H, S, cu, 0.3, 0.5)
    for b, (lo, hi) in enumerate(((0, 9), (9, 23))):
        N = hi - lo
        rank = lambda v, i: sum(1 for j in range(lo, hi) if (v[j], j) < (v[i], i))   # lexicographic
        nl, nh = int(0.3 * N), int(0.5 * N)
        lowH = {i for i in range(lo, hi) if rank(H, i) < nl}
        highH = {i for i in range(lo, hi) if rank(H, i) >= N - nh}
        lowS = {i for i in range(lo, hi) if rank(S, i) < nl}
        highS = {i for i in range(lo, hi) if rank(S, i) >= N - nh}
        assert got[b].tolist() == [len(highH), len(highH & lowS), len(lowH), len(lowH & highS)]


def test_sjf_padding_by_hand():
    y = [5, 1, 9, 2]
    # arrival order, batches of 2: (5,1) max 5, (9,2) max 9
    assert oracle.sjf_padding(y, None, 2) == (4 + 7, 17, (5 + 1) + (2 * 5 + 11))
    # shortest first: (1,2) max 2, (5,9) max 9
    assert oracle.sjf_padding(y, [1, 3, 0, 2], 2) == (1 + 4, 17, (1 + 2) + (2 * 2 + 14))
    # a ragged last batch
    assert oracle.sjf_padding([3, 3, 3], None, 2) == (0, 9, (3 + 3) + (3 + 3))


def test_head_loss_soft_labels_by_hand():
    # a = act(0) = 0 so o = b2 = (0, ln 2, 0): p-hat = (1, 2, 1) / 4.  y = 5 sits in bin 0, so the
    # Eq. 6 targets are (1, e^-1, e^-2) / (1 + e^-1 + e^-2); y-hat = p-hat . c
    h = np.zeros((1, 3))
    W1 = np.zeros((2, 3)); b1 = np.zeros(2); W2 = np.zeros((3, 2)); b2 = np.array([0.0, math.log(2.0), 0.0])
    edges = np.array([0.0, 10.0, 20.0, 30.0]); c = np.array([5.0, 15.0, 25.0])
    lam = 0.7
    loss, _ = oracle.head_loss_and_grads(h, [5.0], edges, c, W1, b1, W2, b2, lam)
    q = np.array([1.0, math.exp(-1.0), math.exp(-2.0)]); q /= q.sum()
    ph = np.array([0.25, 0.5, 0.25])
    ce = -(q * np.log(ph)).sum()
    yhat = (ph * c).sum()
    assert loss == pytest.approx(lam * ce + (1 - lam) * (5.0 - yhat) ** 2, rel=1e-14)
