"""fp32-input paths vs the fp64 oracle, element by element, through the C ABI.

The Tiny configuration states fp32 hidden states, LM-head weights, queries
and keys; these calls then run fp32 kernels (register-tiled VALU code: on
gfx950 the fp32 vector and matrix-core rates are equal) instead of rounding
the inputs to bf16.

Tolerances: with fp32 operands the only errors are fp32 rounding of the dot
products (relative ~sqrt(k) 2^-24 of sum |a b| for k terms) and of exp2 /
log2 (a few ulp), so they are set well inside the bf16 bounds: entropy
|dH| <= 1e-4 nats (bf16: 2e-3), importance |dS| <= 2e-4 S (bf16: 1e-3; the
sharp-attention case multiplies the score error by its query scale of 6),
pooled relative L2 <= 1e-5.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15592_amd as estp
import synth
from synth import inputs as I
from tests._util import check_vocab_argmax, dev, host, rel_l2

pytestmark = pytest.mark.gpu

H_TOL_F32 = 1e-4
S_RTOL_F32 = 2e-4
POOL_RTOL_F32 = 1e-5


def _hidden(n, d, seed):
    g = np.random.default_rng(seed)
    z = g.standard_normal((n, d)).astype(np.float32)
    return (z / np.sqrt((z * z).mean(axis=1, keepdims=True))).astype(np.float32)


def _weight(V, d, seed, std=0.02):
    return (np.random.default_rng(seed).standard_normal((V, d)) * std).astype(np.float32)


ENTROPY_F32_CASES = [
    # (n_tok, d, V, W std, tag)
    (128, 64, 1000, 0.02, "tiny-shape"),
    (1, 8, 7, 0.02, "one-token-width-8"),
    (300, 40, 2500, 0.02, "width-40-partial-stage"),
    (257, 64, 129, 0.02, "vocab-one-past-tile"),
    (700, 256, 5000, 0.02, "several-tiles-per-slice"),
    (129, 4096, 3000, 0.02, "llama-width"),
    (200, 256, 3000, 1.5, "sharp-logits"),
    (64, 128, 600, 0.0, "uniform-logits"),
]


@pytest.mark.parametrize("n,d,V,std,tag", ENTROPY_F32_CASES, ids=[c[-1] for c in ENTROPY_F32_CASES])
def test_entropy_f32_parity(n, d, V, std, tag):
    X = _hidden(n, d, 1)
    W = _weight(V, d, 2, std)
    Xd, Wd = dev(X), dev(W)
    H = host(estp.token_entropy(Xd, Wd))
    ref = oracle.token_entropy(X, W)
    err = np.abs(H.astype(np.float64) - ref)
    print(f"{tag}: max |dH| = {err.max():.3e} nats")
    assert err.max() <= H_TOL_F32
    if std == 0.0:
        np.testing.assert_allclose(H, np.log(V), rtol=0, atol=H_TOL_F32)
    # the most probable next token from the same call: H unchanged, the mode exact (margin rule)
    am = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    np.testing.assert_array_equal(host(estp.token_entropy(Xd, Wd, vocab_argmax=am)), H)
    am = host(am)
    counts = check_vocab_argmax(am, X, W)
    print(f"{tag}: vocab argmax exact on {counts['exact']} rows, near ties {counts['tie']}")
    if std == 0.0:
        assert np.all(am == 0)


def test_entropy_f32_repeatable_bitwise():
    Xd, Wd = dev(_hidden(700, 256, 3)), dev(_weight(5000, 256, 4))
    a = estp.token_entropy(Xd, Wd).clone()
    b = estp.token_entropy(Xd, Wd)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


IMPORTANCE_F32_CASES = [
    # (lengths, L, Hq, Hkv, dh, q scale, tag)
    ([128], 1, 2, 2, 32, 1.0, "tiny-shape"),
    ([1, 5, 31, 32, 33, 64, 65, 130, 257], 2, 4, 2, 64, 1.0, "varlen-ragged-gqa2"),
    ([100, 300], 1, 12, 2, 128, 1.0, "qwen-heads-gqa6"),
    ([200, 77], 2, 8, 2, 128, 6.0, "sharp-attention"),
    ([1], 3, 2, 1, 32, 1.0, "single-token"),
]


def _qk(lengths, L, Hq, Hkv, dh, qscale, seed):
    g = np.random.default_rng(seed)
    n = sum(lengths)
    hs = g.uniform(0.5, 2.0, size=(L, 1, Hq, 1)).astype(np.float32)
    Q = (g.standard_normal((L, n, Hq, dh)).astype(np.float32) * hs * qscale).astype(np.float32)
    K = g.standard_normal((L, n, Hkv, dh)).astype(np.float32)
    return Q, K, I.cu_seqlens_from_lengths(lengths)


@pytest.mark.parametrize("lengths,L,Hq,Hkv,dh,qs,tag", IMPORTANCE_F32_CASES, ids=[c[-1] for c in IMPORTANCE_F32_CASES])
def test_importance_f32_parity(lengths, L, Hq, Hkv, dh, qs, tag):
    Q, K, cu = _qk(lengths, L, Hq, Hkv, dh, qs, 5)
    Qd, Kd, cud = dev(Q), dev(K), dev(cu)
    ref = oracle.attn_importance(Q, K, cu)
    S = host(estp.attn_importance(Qd, Kd, cud, max(lengths)))
    print(f"{tag}: max rel |dS| = {(np.abs(S - ref) / ref).max():.3e}")
    assert np.all(np.abs(S - ref) <= S_RTOL_F32 * ref + 1e-12)
    for b in range(len(lengths)):
        assert abs(S[cu[b]:cu[b + 1]].sum() - L) <= 1e-5 * L
    # the prefill's row normalisers in place of pass 1
    lse = dev(oracle.attn_row_lse(Q, K, cu).astype(np.float32))
    S2 = host(estp.attn_importance_from_lse(Qd, Kd, lse, cud, max(lengths)))
    assert np.all(np.abs(S2 - ref) <= S_RTOL_F32 * ref + 1e-12)
    # diagonal left out and per-layer weights
    w = [1.5 - 0.75 * l for l in range(L)]
    ref_both = oracle.attn_importance(Q, K, cu, exclude_self=True, layer_weights=w)
    tol = S_RTOL_F32 * np.abs(ref_both) + 1e-6 * np.abs(ref_both).max()
    for kw in ({}, {"lse": lse}):
        got = host(estp.attn_importance_ex(Qd, Kd, cud, max(lengths), exclude_self=True, layer_weights=w, **kw))
        assert np.all(np.abs(got - ref_both) <= tol)


def test_importance_f32_repeatable_bitwise():
    Q, K, cu = _qk([300, 45, 600], 2, 8, 2, 128, 1.0, 6)
    Qd, Kd, cud = dev(Q), dev(K), dev(cu)
    a = estp.attn_importance(Qd, Kd, cud, 600).clone()
    b = estp.attn_importance(Qd, Kd, cud, 600)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_importance_f32_live_block_list():
    # many short prompts and one long one: both passes run over the list of live 256-row blocks
    lengths = [3] * 40 + [700] + [17] * 9
    Q, K, cu = _qk(lengths, 1, 4, 2, 64, 1.0, 8)
    S = host(estp.attn_importance(dev(Q), dev(K), dev(cu), max(lengths)))
    ref = oracle.attn_importance(Q, K, cu)
    assert np.all(np.abs(S - ref) <= S_RTOL_F32 * ref + 1e-12)


def test_path_f32_tiny_end_to_end():
    # the Tiny configuration as stated: fp32 inputs end to end
    w = synth.get_workload("tiny")
    assert w.dtype == "f32"
    inp = I.make_inputs(w, 42)
    cu = inp["cu_seqlens"]
    head = (inp["W1"], inp["b1"], inp["W2"], inp["b2"], inp["centres"])
    out = estp.run_path(dev(inp["X"]), dev(inp["W"]), dev(inp["Q"]), dev(inp["K"]), dev(cu), int(w.seq_len),
                        0.5, 0.5, 1.0, "none", head=tuple(dev(t) for t in head[:4]) + (None,))
    torch.cuda.synchronize()
    ref = oracle.run_path(inp["X"], inp["W"], inp["Q"], inp["K"], cu, 0.5, 0.5, 1.0, "none", head=head)
    assert np.abs(host(out["H"]).astype(np.float64) - ref["H"]).max() <= H_TOL_F32
    S = host(out["S"])
    assert np.all(np.abs(S - ref["S"]) <= S_RTOL_F32 * ref["S"] + 1e-12)
    assert rel_l2(host(out["pooled"]), ref["pooled"]) <= POOL_RTOL_F32
    np.testing.assert_allclose(host(out["yhat"]), ref["yhat"], rtol=1e-4, atol=1e-6)
