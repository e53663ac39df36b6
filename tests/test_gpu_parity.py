"""HIP path vs the fp64 oracle, element by element, through the C ABI.

Tolerances (fixed by the targets of the path): entropy |dH| <= 2e-3 nats;
importance |dS| <= 1e-3 S + 1e-12; pooled vectors relative L2 <= 1e-3 per
prompt; length head relative 1e-3; indices exact outside near ties (margin
rule, see tests/_util.py).  Inputs are bf16 (the oracle widens the same bits).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15592_amd as estp
import synth
from synth import inputs as I
from tests._util import check_argmax_margin, check_order_margin, check_vocab_argmax, dev, host, rel_l2

pytestmark = pytest.mark.gpu

H_TOL = 2e-3
S_RTOL = 1e-3
POOL_RTOL = 1e-3


def _bf16(a):
    return I.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def _hidden(n, d, seed, scale=1.0):
    g = np.random.default_rng(seed)
    z = g.standard_normal((n, d)).astype(np.float32)
    z /= np.sqrt((z * z).mean(axis=1, keepdims=True))
    return _bf16(z * scale)


def _weight(V, d, seed, std=0.02):
    g = np.random.default_rng(seed)
    return _bf16(g.standard_normal((V, d)).astype(np.float32) * std)


# ------------------------------------------------------------------------------------------ entropy

ENTROPY_CASES = [
    # (n_tok, d, V, W std, tag)
    (128, 64, 1000, 0.02, "tiny-shape"),
    (1, 64, 7, 0.02, "one-token-seven-words"),
    (300, 128, 2500, 0.02, "ragged-tokens-and-vocab"),
    (513, 1536, 4099, 0.02, "qwen-width-ragged"),
    (256, 4096, 32768, 0.02, "llama-width-16-slices"),
    (200, 256, 3000, 1.5, "sharp-logits"),
    (64, 128, 600, 0.0, "uniform-logits"),
    # widths that are an odd multiple of 32 take the 32-deep staging
    (77, 32, 1300, 0.02, "width-32"),
    (300, 96, 2500, 0.02, "width-96-ragged"),
    (130, 4128, 3000, 0.02, "width-4128"),
    # tile edges: one vocabulary row, exactly one 256 x 256 tile, one past it
    (5, 64, 1, 0.02, "one-word-vocab"),
    (256, 64, 256, 0.02, "exact-tile"),
    (257, 64, 257, 0.02, "tile-plus-one"),
]


@pytest.mark.parametrize("n_tok,d,V,std,tag", ENTROPY_CASES, ids=[c[-1] for c in ENTROPY_CASES])
def test_entropy_parity(n_tok, d, V, std, tag):
    X = _hidden(n_tok, d, 1)
    W = _weight(V, d, 2, std)
    Xd, Wd = dev(X), dev(W)
    H = host(estp.token_entropy(Xd, Wd))
    ref = oracle.token_entropy(X, W)
    err = np.abs(H - ref).max()
    print(f"{tag}: max |dH| = {err:.3e} nats (H in [{ref.min():.3f}, {ref.max():.3f}])")
    assert err <= H_TOL
    if std == 0.0:
        np.testing.assert_allclose(H, math.log(V), atol=H_TOL)
    # the same call asked for the most probable next token as well: H unchanged bit for bit,
    # the mode exact under the margin rule
    am = torch.full((n_tok,), -7, dtype=torch.int32, device="cuda")
    H2 = host(estp.token_entropy(Xd, Wd, vocab_argmax=am))
    np.testing.assert_array_equal(H2, H)
    am = host(am)
    counts = check_vocab_argmax(am, X, W)
    print(f"{tag}: vocab argmax exact on {counts['exact']} rows, near ties {counts['tie']}")
    if std == 0.0:
        assert np.all(am == 0)  # every logit exactly 0: the lowest index


def test_entropy_argmax_exact_ties():
    # copies of one strong row at several vocabulary positions tie exactly (identical operands give
    # identical sums): the lowest position wins, in whichever tile, half or slice the copies land
    n_tok, d, V = 300, 256, 9000
    X = _hidden(n_tok, d, 7)
    W = _weight(V, d, 8)
    g = np.random.default_rng(9)
    strong = _bf16(g.standard_normal(d).astype(np.float32) * 0.3)
    for pos in (8700, 4100, 300, 129, 7000):
        W[pos] = strong
    am = torch.empty(n_tok, dtype=torch.int32, device="cuda")
    estp.token_entropy(dev(X), dev(W), vocab_argmax=am)
    am = host(am)
    z = oracle.widen(X) @ oracle.widen(strong)
    rows = z > (oracle.widen(X) @ oracle.widen(np.delete(W, [8700, 4100, 300, 129, 7000], axis=0)).T).max(axis=1) + 0.1
    assert rows.sum() > 50
    assert np.all(am[rows] == 129), np.unique(am[rows])
    check_vocab_argmax(am, X, W)


def test_entropy_late_peak():
    # weight rows scaled up along the vocabulary: the first tiles hold only small logits, so
    # later tiles exceed the running reference by far more than 2^64 in weight and are
    # refolded exactly with their own max (the ragged last tile always is)
    n_tok, d, V = 300, 256, 12000
    X = _hidden(n_tok, d, 5)
    step = np.where(np.arange(V) < 7000, 0.05, 80.0).astype(np.float32)[:, None]
    W = _bf16(np.random.default_rng(6).standard_normal((V, d)).astype(np.float32) * 0.02 * step)
    H = host(estp.token_entropy(dev(X), dev(W)))
    ref = oracle.token_entropy(X, W)
    logits = oracle.widen(X)[:4] @ oracle.widen(W).T
    print(f"late peak: logit range of the first tile {np.abs(logits[:, :256]).max():.1f}, "
          f"overall {np.abs(logits).max():.1f}; max |dH| = {np.abs(H - ref).max():.3e}")
    assert np.abs(H - ref).max() <= H_TOL


def test_entropy_repeatable_bitwise():
    X = dev(_hidden(700, 256, 3))
    W = dev(_weight(5000, 256, 4))
    a = estp.token_entropy(X, W).clone()
    b = estp.token_entropy(X, W)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_entropy_rejects_bf16_width_not_multiple_of_32():
    X = torch.zeros(4, 40, device="cuda", dtype=torch.bfloat16)
    W = torch.zeros(10, 40, device="cuda", dtype=torch.bfloat16)
    with pytest.raises(estp.EstpError) as ei:
        estp.token_entropy(X, W)
    assert ei.value.status == 2


# ------------------------------------------------------------------------------------------ importance

IMPORTANCE_CASES = [
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
    Q = _bf16(g.standard_normal((L, n, Hq, dh)).astype(np.float32) * hs * qscale)
    K = _bf16(g.standard_normal((L, n, Hkv, dh)).astype(np.float32))
    cu = I.cu_seqlens_from_lengths(lengths)
    return Q, K, cu


@pytest.mark.parametrize("lengths,L,Hq,Hkv,dh,qs,tag", IMPORTANCE_CASES, ids=[c[-1] for c in IMPORTANCE_CASES])
def test_importance_parity(lengths, L, Hq, Hkv, dh, qs, tag):
    Q, K, cu = _qk(lengths, L, Hq, Hkv, dh, qs, 5)
    S = host(estp.attn_importance(dev(Q), dev(K), dev(cu), max(lengths)))
    ref = oracle.attn_importance(Q, K, cu)
    rel = np.abs(S - ref) / ref
    print(f"{tag}: max rel |dS| = {rel.max():.3e}")
    assert np.all(np.abs(S - ref) <= S_RTOL * ref + 1e-12)
    for b in range(len(lengths)):
        assert abs(S[cu[b]:cu[b + 1]].sum() - L) <= 1e-4 * L


@pytest.mark.parametrize("lengths,L,Hq,Hkv,dh,qs,tag", IMPORTANCE_CASES, ids=[c[-1] for c in IMPORTANCE_CASES])
def test_importance_from_lse_parity(lengths, L, Hq, Hkv, dh, qs, tag):
    # the prefill's row normalisers (here the oracle's) replace pass 1
    Q, K, cu = _qk(lengths, L, Hq, Hkv, dh, qs, 5)
    lse = oracle.attn_row_lse(Q, K, cu)
    S = host(estp.attn_importance_from_lse(dev(Q), dev(K), dev(lse.astype(np.float32)), dev(cu), max(lengths)))
    ref = oracle.attn_importance(Q, K, cu)
    print(f"{tag}: max rel |dS| = {(np.abs(S - ref) / ref).max():.3e}")
    assert np.all(np.abs(S - ref) <= S_RTOL * ref + 1e-12)


def test_importance_from_lse_uses_the_given_normalisers():
    # normalisers off by a per-row shift scale each row: the result follows the given lse
    Q, K, cu = _qk([70, 260, 9], 2, 4, 2, 64, 1.0, 12)
    shifted = oracle.attn_row_lse(Q, K, cu) + np.random.default_rng(13).uniform(-0.5, 0.5, size=(2, 4, 339))
    S = host(estp.attn_importance_from_lse(dev(Q), dev(K), dev(shifted.astype(np.float32)), dev(cu), 260))
    ref = oracle.attn_importance_from_lse(Q, K, cu, shifted.astype(np.float32))
    assert np.all(np.abs(S - ref) <= S_RTOL * ref + 1e-12)
    assert not np.allclose(ref, oracle.attn_importance(Q, K, cu), rtol=1e-2)


@pytest.mark.parametrize("lengths,L,Hq,Hkv,dh,qs,tag", IMPORTANCE_CASES, ids=[c[-1] for c in IMPORTANCE_CASES])
def test_importance_ex_variants_parity(lengths, L, Hq, Hkv, dh, qs, tag):
    # diagonal left out of the column sums, per-layer weights, with and without given row LSEs
    Q, K, cu = _qk(lengths, L, Hq, Hkv, dh, qs, 5)
    Qd, Kd, cud = dev(Q), dev(K), dev(cu)
    w = [1.5 - 0.75 * l for l in range(L)]
    ref_ex = oracle.attn_importance(Q, K, cu, exclude_self=True)
    ref_w = oracle.attn_importance(Q, K, cu, layer_weights=w)
    ref_both = oracle.attn_importance(Q, K, cu, exclude_self=True, layer_weights=w)
    lse = dev(oracle.attn_row_lse(Q, K, cu).astype(np.float32))
    tol = lambda ref: S_RTOL * np.abs(ref) + 1e-6 * np.abs(ref).max()
    for with_lse in (False, True):
        kw = {"lse": lse} if with_lse else {}
        got = host(estp.attn_importance_ex(Qd, Kd, cud, max(lengths), exclude_self=True, **kw))
        assert np.all(np.abs(got - ref_ex) <= tol(ref_ex))
        got = host(estp.attn_importance_ex(Qd, Kd, cud, max(lengths), layer_weights=w, **kw))
        assert np.all(np.abs(got - ref_w) <= tol(ref_w))
        got = host(estp.attn_importance_ex(Qd, Kd, cud, max(lengths), layer_weights=w, exclude_self=True, **kw))
        assert np.all(np.abs(got - ref_both) <= tol(ref_both))
    # with no variant the extended call is the plain one
    plain = host(estp.attn_importance(Qd, Kd, cud, max(lengths)))
    assert np.array_equal(host(estp.attn_importance_ex(Qd, Kd, cud, max(lengths))), plain)


@pytest.mark.parametrize("f32", [False, True], ids=["bf16", "f32"])
def test_importance_accepts_a_larger_max_seqlen(f32):
    # max_seqlen is an upper bound on the prompt lengths (at most n_tok): a looser one changes the
    # grids (blocks past every prompt, the list of live blocks, the head split) but not the result
    Q, K, cu = _qk([70, 1100, 9, 300], 2, 4, 2, 64, 1.0, 21)
    if f32:
        Q, K = oracle.widen(Q).astype(np.float32), oracle.widen(K).astype(np.float32)
    ref = oracle.attn_importance(Q, K, cu)
    for max_seqlen in (1100, 1300, 1479):
        S = host(estp.attn_importance(dev(Q), dev(K), dev(cu), max_seqlen))
        assert np.all(np.abs(S - ref) <= S_RTOL * ref + 1e-12), max_seqlen


def test_importance_repeatable_bitwise():
    Q, K, cu = _qk([300, 45, 600], 2, 8, 2, 128, 1.0, 6)
    Qd, Kd, cud = dev(Q), dev(K), dev(cu)
    a = estp.attn_importance(Qd, Kd, cud, 600).clone()
    b = estp.attn_importance(Qd, Kd, cud, 600)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# ------------------------------------------------------------------------------------------ combine + pool

COMBINE_GRID = [(0.1, 0.9, 1.0), (0.5, 0.5, 0.5), (0.9, 0.1, 2.0), (0.0, 0.0, 1.0), (1.0, 0.0, 1.0), (0.0, 1.0, 0.5)]


@pytest.mark.parametrize("xdtype", ["bf16", "f32"])
@pytest.mark.parametrize("norm", ["none", "zscore", "minmax"])
def test_combine_pool_parity(xdtype, norm):
    lengths = [1, 7, 256, 257, 600, 33]
    n = sum(lengths)
    d = 520
    g = np.random.default_rng(7)
    Xf = g.standard_normal((n, d)).astype(np.float32)
    X = _bf16(Xf) if xdtype == "bf16" else Xf
    S = (g.random(n) / 50).astype(np.float32)
    Hh = (g.random(n) * 8).astype(np.float32)
    cu = I.cu_seqlens_from_lengths(lengths)
    Xd, Sd, Hd, cud = dev(X), dev(S), dev(Hh), dev(cu)
    ties = 0
    for l1, l2, a in COMBINE_GRID:
        pooled, e, top = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm)
        e_ref, top_ref = oracle.combine_weights(S, Hh, cu, l1, l2, a, norm)
        p_ref = oracle.pool(X, e_ref, cu)
        np.testing.assert_allclose(host(e), e_ref, rtol=1e-4, atol=1e-12)
        P = host(pooled)
        top = host(top)
        for b in range(len(lengths)):
            assert rel_l2(P[b], p_ref[b]) <= POOL_RTOL
            lo, hi = cu[b], cu[b + 1]
            res = check_argmax_margin(int(top[b]) - lo, e_ref[lo:hi], 1e-5 * e_ref[lo:hi].max())
            ties += res == "tie"
    print(f"{xdtype}/{norm}: near-tie top groups seen: {ties}")


def test_combine_pool_special_cases():
    # lambda = 0 -> average pooling; identical rows pool to that row
    lengths = [5, 300]
    n = sum(lengths)
    g = np.random.default_rng(8)
    X = _bf16(g.standard_normal((n, 64)))
    cu = I.cu_seqlens_from_lengths(lengths)
    S = g.random(n).astype(np.float32)
    H = g.random(n).astype(np.float32)
    pooled, e, _ = estp.combine_pool(dev(X), dev(S), dev(H), dev(cu), 300, 0.0, 0.0, 1.0)
    Xw = oracle.widen(X)
    for b in range(2):
        np.testing.assert_allclose(host(e)[cu[b]:cu[b + 1]], 1.0 / lengths[b], rtol=1e-6)
        assert rel_l2(host(pooled)[b], Xw[cu[b]:cu[b + 1]].mean(0)) <= 1e-5
    Xs = np.tile(X[:1], (n, 1))
    pooled, _, _ = estp.combine_pool(dev(Xs), dev(S), dev(H), dev(cu), 300, 0.7, 0.3, 0.5)
    for b in range(2):
        assert rel_l2(host(pooled)[b], Xw[0]) <= 1e-6


def test_combine_pool_slices_and_reused_workspace():
    # three feature slices (the last one ragged), a prompt of many chunks, and one
    # workspace shared by consecutive calls (its arrival counters must come back clean)
    lengths = [5000, 3, 1300]
    n = sum(lengths)
    d = 4616
    g = np.random.default_rng(10)
    X = _bf16(g.standard_normal((n, d)).astype(np.float32))
    S = (g.random(n) / 20).astype(np.float32)
    Hh = (g.random(n) * 8).astype(np.float32)
    cu = I.cu_seqlens_from_lengths(lengths)
    Xd, Sd, Hd, cud = dev(X), dev(S), dev(Hh), dev(cu)
    nb = estp.load().estp_combine_pool_workspace_size(n, len(lengths), max(lengths), d, 0)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    for l1, l2, a, norm in [(0.5, 0.5, 1.0, "none"), (0.9, 0.1, 0.5, "zscore"), (0.2, 0.8, 2.0, "none")]:
        pooled, e, top = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm, workspace=ws)
        e_ref, _ = oracle.combine_weights(S, Hh, cu, l1, l2, a, norm)
        p_ref = oracle.pool(X, e_ref, cu)
        np.testing.assert_allclose(host(e), e_ref, rtol=1e-4, atol=1e-12)
        P = host(pooled)
        top = host(top)
        for b in range(len(lengths)):
            assert rel_l2(P[b], p_ref[b]) <= POOL_RTOL
            lo, hi = cu[b], cu[b + 1]
            check_argmax_margin(int(top[b]) - lo, e_ref[lo:hi], 1e-5 * e_ref[lo:hi].max())


@pytest.mark.parametrize("xdtype,d,spread,norm", [("bf16", 2040, 10, "none"), ("bf16", 4096, 0, "zscore"),
                                                 ("f32", 1000, 3, "minmax")])
def test_combine_pool_equal_prompts_one_kernel(xdtype, d, spread, norm):
    # prompts of (nearly) equal length whose (prompt, 512-feature slice) workgroups fill
    # every compute unit four times over: the one-kernel whole-prompt pooling path
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    slices = (d + 511) // 512
    B = -(-4 * n_cu // slices)
    g = np.random.default_rng(12 + d)
    lengths = (100 - g.integers(0, spread + 1, size=B)).tolist()
    n = sum(lengths)
    Xf = g.standard_normal((n, d)).astype(np.float32)
    X = _bf16(Xf) if xdtype == "bf16" else Xf
    S = (g.random(n) / 30).astype(np.float32)
    Hh = (g.random(n) * 8).astype(np.float32)
    cu = I.cu_seqlens_from_lengths(lengths)
    Xd, Sd, Hd, cud = dev(X), dev(S), dev(Hh), dev(cu)
    for l1, l2, a in [(0.5, 0.5, 1.0), (0.9, 0.1, 0.5)]:
        pooled, e, top = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm)
        e_ref, _ = oracle.combine_weights(S, Hh, cu, l1, l2, a, norm)
        p_ref = oracle.pool(X, e_ref, cu)
        np.testing.assert_allclose(host(e), e_ref, rtol=1e-4, atol=1e-12)
        P, top = host(pooled), host(top)
        for b in range(B):
            assert rel_l2(P[b], p_ref[b]) <= POOL_RTOL
            lo, hi = cu[b], cu[b + 1]
            check_argmax_margin(int(top[b]) - lo, e_ref[lo:hi], 1e-5 * e_ref[lo:hi].max())
        again, _, _ = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm)
        assert torch.equal(again, pooled)
        # without the optional weights and top-token outputs
        bare, e0, t0 = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm, want_e=False, want_top=False)
        assert e0 is None and t0 is None and torch.equal(bare, pooled)


def test_combine_pool_many_short_prompts():
    # one long prompt and 299 short ones: the pooling runs over the list of live chunks
    # (the full prompt x chunk grid would be mostly empty), built by a scan over prompts
    g = np.random.default_rng(11)
    lengths = [2000] + g.integers(1, 41, size=299).tolist()
    n = sum(lengths)
    d = 4096
    X = _bf16(g.standard_normal((n, d)).astype(np.float32))
    S = (g.random(n) / 20).astype(np.float32)
    Hh = (g.random(n) * 8).astype(np.float32)
    cu = I.cu_seqlens_from_lengths(lengths)
    pooled, e, top = estp.combine_pool(dev(X), dev(S), dev(Hh), dev(cu), max(lengths), 0.6, 0.4, 1.0, "zscore")
    e_ref, _ = oracle.combine_weights(S, Hh, cu, 0.6, 0.4, 1.0, "zscore")
    p_ref = oracle.pool(X, e_ref, cu)
    np.testing.assert_allclose(host(e), e_ref, rtol=1e-4, atol=1e-12)
    P, top = host(pooled), host(top)
    for b in range(len(lengths)):
        assert rel_l2(P[b], p_ref[b]) <= POOL_RTOL
        lo, hi = cu[b], cu[b + 1]
        check_argmax_margin(int(top[b]) - lo, e_ref[lo:hi], 1e-5 * e_ref[lo:hi].max())


POOL_PATH_CASES = [
    # (lengths, d, dtype, tag): which pooling kernel a batch takes follows from its shape
    ("mixed-1-3000", 8200, "bf16", "one-kernel, width 8200: four minimum slices"),
    ("many-1-20", 128, "bf16", "one-kernel, 3000 prompts in the in-kernel scan"),
    ("mixed-1-3000", 1000, "f32", "one-kernel, fp32 hidden states"),
    ([9000, 5, 300], 264, "bf16", "chunked (prompt over 8192 rows), list of live chunks"),
    ([8500, 8400], 136, "f32", "chunked, full prompt x chunk grid"),
    ("many-1-3", 64, "bf16", "chunked (over 8192 prompts), list of live chunks"),
    ("n8192-1-4", 72, "bf16", "one-kernel, 8192 prompts: the in-kernel scan's limit"),
    ("n8193-1-4", 72, "bf16", "chunked, one prompt past the in-kernel scan's limit"),
]


def _pool_lengths(spec, g):
    if spec == "mixed-1-3000":
        return [3000, 1, 2] + np.exp(g.uniform(0, np.log(3000), size=21)).astype(int).tolist()
    if spec == "many-1-20":
        return g.integers(1, 21, size=3000).tolist()
    if spec == "many-1-3":
        return g.integers(1, 4, size=9000).tolist()
    if isinstance(spec, str) and spec.startswith("n") and spec.endswith("-1-4"):
        return g.integers(1, 5, size=int(spec[1:-4])).tolist()
    return list(spec)


@pytest.mark.parametrize("spec,d,xdtype,tag", POOL_PATH_CASES, ids=[c[-1] for c in POOL_PATH_CASES])
def test_combine_pool_paths(spec, d, xdtype, tag):
    g = np.random.default_rng(len(tag) + d)
    lengths = _pool_lengths(spec, g)
    n = sum(lengths)
    Xf = g.standard_normal((n, d)).astype(np.float32)
    X = _bf16(Xf) if xdtype == "bf16" else Xf
    S = (g.random(n) / 20).astype(np.float32)
    Hh = (g.random(n) * 8).astype(np.float32)
    cu = I.cu_seqlens_from_lengths(lengths)
    Xd, Sd, Hd, cud = dev(X), dev(S), dev(Hh), dev(cu)
    for l1, l2, a, norm in [(0.5, 0.5, 1.0, "none"), (0.8, 0.2, 0.5, "zscore")]:
        pooled, e, top = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm)
        e_ref, _ = oracle.combine_weights(S, Hh, cu, l1, l2, a, norm)
        p_ref = oracle.pool(X, e_ref, cu)
        np.testing.assert_allclose(host(e), e_ref, rtol=1e-4, atol=1e-12)
        P, top = host(pooled), host(top)
        errs = [rel_l2(P[b], p_ref[b]) for b in range(len(lengths))]
        print(f"{tag}: {len(lengths)} prompts, max pooled rel L2 {max(errs):.1e}")
        assert max(errs) <= POOL_RTOL
        for b in range(len(lengths)):
            lo, hi = cu[b], cu[b + 1]
            check_argmax_margin(int(top[b]) - lo, e_ref[lo:hi], 1e-5 * e_ref[lo:hi].max())
        again, _, _ = estp.combine_pool(Xd, Sd, Hd, cud, max(lengths), l1, l2, a, norm)
        assert torch.equal(again, pooled)


def test_combine_pool_accepts_a_larger_max_seqlen():
    # a looser bound on the prompt lengths moves the call to another pooling kernel (whole prompt,
    # length-sized slices, chunked), each within the bound of the oracle
    g = np.random.default_rng(31)
    lengths = [700, 650, 690, 710] * 8  # 32 prompts x 8 slices of 512 features: one per compute unit
    n, d = sum(lengths), 4096
    X = _bf16(g.standard_normal((n, d)).astype(np.float32))
    S = (g.random(n) / 20).astype(np.float32)
    Hh = (g.random(n) * 8).astype(np.float32)
    cu = I.cu_seqlens_from_lengths(lengths)
    e_ref, _ = oracle.combine_weights(S, Hh, cu, 0.5, 0.5, 1.0, "none")
    p_ref = oracle.pool(X, e_ref, cu)
    for max_seqlen in (710, 4000, 9000):
        pooled, e, _ = estp.combine_pool(dev(X), dev(S), dev(Hh), dev(cu), max_seqlen, 0.5, 0.5, 1.0, "none")
        np.testing.assert_allclose(host(e), e_ref, rtol=1e-4, atol=1e-12)
        P = host(pooled)
        assert max(rel_l2(P[b], p_ref[b]) for b in range(len(lengths))) <= POOL_RTOL, max_seqlen


# ------------------------------------------------------------------------------------------ length head

@pytest.mark.parametrize("K,act,B,d,Hdn", [(1, "relu", 37, 256, 96), (8, "relu", 37, 256, 96),
                                          (8, "gelu_tanh", 37, 256, 96), (1, "gelu_tanh", 37, 256, 96),
                                          (1, "relu", 70, 1000, 1024), (16, "relu", 3, 4096, 40)])
def test_predict_parity(K, act, B, d, Hdn):
    g = np.random.default_rng(9)
    P = g.standard_normal((B, d)).astype(np.float32)
    W1 = (g.standard_normal((Hdn, d)) * 0.1).astype(np.float32)
    b1 = (g.standard_normal(Hdn) * 0.1).astype(np.float32)
    W2 = (g.standard_normal((K, Hdn)) * 0.3).astype(np.float32)
    b2 = (g.standard_normal(K) * 0.1).astype(np.float32)
    c = np.linspace(50, 3000, K).astype(np.float32)
    y, bins, order = estp.predict(dev(P), dev(W1), dev(b1), dev(W2), dev(b2), dev(c) if K > 1 else None, act)
    y_ref, bin_ref, order_ref = oracle.predict(P, W1, b1, W2, b2, c, act)
    y = host(y)
    np.testing.assert_allclose(y, y_ref, rtol=1e-3, atol=1e-5)
    delta = 4e-3 * np.abs(y_ref) + 4e-5
    ties = check_order_margin(host(order), y_ref, delta)
    if K > 1:
        h = np.asarray(P, np.float64)
        a = h @ W1.T + b1
        a = np.maximum(a, 0) if act == "relu" else 0.5 * a * (1 + np.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3)))
        o = a @ W2.T + b2
        for b in range(B):
            check_argmax_margin(int(host(bins)[b]), o[b], 4e-3 * np.abs(o[b]).max())
    print(f"K={K} {act}: max rel dy = {np.max(np.abs(y - y_ref) / np.abs(y_ref)):.2e}, near-tie order pairs {ties}")


# ------------------------------------------------------------------------------------------ whole path

def _run_both(w, seed=42, lam=(0.5, 0.5), alpha=1.0, norm="none"):
    inp = I.make_inputs(w, seed)
    if w.dtype == "f32":  # the matrix-core kernels take bf16: round once, both sides see the same bits
        for k in ("X", "W", "Q", "K"):
            inp[k] = I.f32_to_bf16_bits(inp[k])
    cu = inp["cu_seqlens"]
    head = (inp["W1"], inp["b1"], inp["W2"], inp["b2"], inp["centres"])
    out = estp.run_path(dev(inp["X"]), dev(inp["W"]), dev(inp["Q"]), dev(inp["K"]), dev(cu), int(inp["lengths"].max()),
                        lam[0], lam[1], alpha, norm, head=tuple(dev(t) for t in head[:4]) + (None,))
    ref = oracle.run_path(inp["X"], inp["W"], inp["Q"], inp["K"], cu, lam[0], lam[1], alpha, norm, head=head)
    return {k: (host(v) if isinstance(v, torch.Tensor) else v) for k, v in out.items()}, ref, cu


def test_full_path_tiny():
    w = synth.get_workload("tiny")
    got, ref, cu = _run_both(w)
    assert np.abs(got["H"] - ref["H"]).max() <= H_TOL
    assert np.all(np.abs(got["S"] - ref["S"]) <= S_RTOL * ref["S"] + 1e-12)
    assert rel_l2(got["pooled"][0], ref["pooled"][0]) <= POOL_RTOL
    np.testing.assert_allclose(got["yhat"], ref["yhat"], rtol=1e-3, atol=1e-6)
    assert list(got["order"]) == list(ref["order"])
    print(f"tiny: |dH| {np.abs(got['H'] - ref['H']).max():.2e}, rel dS "
          f"{(np.abs(got['S'] - ref['S']) / ref['S']).max():.2e}, pooled rel {rel_l2(got['pooled'], ref['pooled']):.2e}")


def test_full_path_qwen_shaped_small():
    # Qwen2.5-1.5B widths and vocabulary (d=1536, V=151936, 12/2 heads of 128), 3 short prompts
    w = synth.get_workload("qwen", n_prompts=3, seq_len=40)
    got, ref, cu = _run_both(w, lam=(0.9, 0.1), alpha=0.5, norm="zscore")
    assert np.abs(got["H"] - ref["H"]).max() <= H_TOL
    assert np.all(np.abs(got["S"] - ref["S"]) <= S_RTOL * ref["S"] + 1e-12)
    for b in range(3):
        assert rel_l2(got["pooled"][b], ref["pooled"][b]) <= POOL_RTOL


# ------------------------------------------------------------------------------------------ head training step

def _train_problem(B, d, Hd, K, seed):
    g = np.random.default_rng(seed)
    h = g.standard_normal((B, d)).astype(np.float32)
    P = {"W1": (g.standard_normal((Hd, d)) * 0.05).astype(np.float32),
         "b1": (g.standard_normal(Hd) * 0.1).astype(np.float32),
         "W2": (g.standard_normal((K, Hd)) * 0.2).astype(np.float32),
         "b2": (g.standard_normal(K) * 0.1).astype(np.float32)}
    edges = np.concatenate([[0.0], np.geomspace(64.0, 16384.0, K)]).astype(np.float32)
    centres = (0.5 * (edges[1:] + edges[:-1])).astype(np.float32)
    y = np.exp(g.uniform(np.log(16.0), np.log(20000.0), size=B)).astype(np.float32)
    return h, y, edges, centres, P


def _flat(P):
    return np.concatenate([P["W1"].ravel(), P["b1"], P["W2"].ravel(), P["b2"]]).astype(np.float32)


def _split(flat, d, Hd, K):
    n1 = Hd * d
    return {"W1": flat[:n1].reshape(Hd, d), "b1": flat[n1:n1 + Hd], "W2": flat[n1 + Hd:n1 + Hd + K * Hd].reshape(K, Hd),
            "b2": flat[n1 + Hd + K * Hd:]}


@pytest.mark.parametrize("act", ["relu", "gelu_tanh"])
@pytest.mark.parametrize("B,d,Hd,K", [(37, 256, 96, 8), (32, 4096, 1024, 16), (5, 1000, 40, 2)])
def test_head_train_step_parity(act, B, d, Hd, K):
    # three AdamW steps on the device; each is checked against one fp64 oracle step taken from
    # the device's own state before it (Adam's g / sqrt(v) turns fp32 noise in near-zero gradients
    # into O(lr) differences, so free-running trajectories are not comparable step for step)
    h, y, edges, centres, P = _train_problem(B, d, Hd, K, 20)
    lam, lr = 0.6, 1e-3
    theta = dev(_flat(P))
    m = torch.zeros_like(theta)
    v = torch.zeros_like(theta)
    hd, yd, ed, cd = dev(h), dev(y), dev(edges), dev(centres)
    for t in (1, 2, 3):
        P0 = _split(host(theta).astype(np.float64), d, Hd, K)
        M0 = _split(host(m).astype(np.float64), d, Hd, K)
        V0 = _split(host(v).astype(np.float64), d, Hd, K)
        loss = host(estp.head_train_step(hd, yd, ed, cd, theta, m, v, Hd, t, lam, lr, act=act))[0]
        ref_loss, g, Pr, Mr, Vr = oracle.head_train_step(h, y, edges, centres, P0, M0, V0, t, lam, lr, act=act)
        assert loss == pytest.approx(ref_loss, rel=1e-3)  # fp32 forward: the squared error amplifies y - yhat cancellation
        cat = lambda D: np.concatenate([D["W1"].ravel(), D["b1"], D["W2"].ravel(), D["b2"]])
        gr, rm, rt = cat(g), cat(Mr), cat(Pr)
        gm, th = host(m), host(theta)
        # the first moments carry this step's gradients
        assert np.abs(gm - rm).max() <= 1e-4 * np.abs(rm).max(), f"step {t}: moment error"
        # AdamW moves a coordinate by about lr g / |g|: where g is resolved above fp32 noise the step
        # matches to 1% of lr; elsewhere its sign is arbitrary but the step stays bounded by ~lr
        big = (np.abs(gr) > 1e-2 * np.abs(gr).max()) | (gr == 0.0)
        err = np.abs(th - rt)
        close = err <= 1e-2 * lr + 1e-6 * np.abs(rt).max()
        print(f"step {t}: resolved {big.mean():.3f}, within 1% of lr {close.mean():.4f}, max err {err.max() / lr:.2f} lr")
        assert close[big].all()
        assert close.mean() > 0.95
        assert err.max() <= 2.5 * lr


def test_head_train_step_matches_predict_and_learns():
    # after training, estp_predict reads its parameters from the same flat vector, and the
    # Eq. 8 loss has gone down on the batch
    B, d, Hd, K = 64, 512, 128, 12
    h, y, edges, centres, P = _train_problem(B, d, Hd, K, 21)
    theta = dev(_flat(P))
    m = torch.zeros_like(theta)
    v = torch.zeros_like(theta)
    hd, yd, ed, cd = dev(h), dev(y), dev(edges), dev(centres)
    losses = []
    for t in range(1, 201):
        losses.append(float(host(estp.head_train_step(hd, yd, ed, cd, theta, m, v, Hd, t, 0.9, 3e-3))[0]))
    assert losses[-1] < 0.7 * losses[0]
    W1, b1, W2, b2 = estp.head_param_views(theta, d, Hd, K)
    yhat, _, _ = estp.predict(hd, W1, b1, W2, b2, cd)
    ref, _, _ = oracle.predict(h, host(W1), host(b1), host(W2), host(b2), centres)
    np.testing.assert_allclose(host(yhat), ref, rtol=1e-4)


# ------------------------------------------------------------------------------------------ analyses

@pytest.mark.parametrize("frac", [(0.4, 0.4), (0.3, 0.5), (0.0, 1.0), (1.0, 0.0)])
def test_misalignment_parity(frac):
    # integer counts: bit-exact against the oracle on the same float32 scores (ties included)
    g = np.random.default_rng(30)
    lengths = [1, 2, 5, 64, 257, 1000, 4096, 33]
    n = sum(lengths)
    H = g.standard_normal(n).astype(np.float32)
    S = (g.integers(0, 40, size=n) / 7.0).astype(np.float32)   # many equal values
    H[100:150] = 0.0
    cu = I.cu_seqlens_from_lengths(lengths)
    got = host(estp.misalignment(dev(H), dev(S), dev(cu), *frac))
    ref = oracle.misalignment_counts(H, S, cu, *frac)
    assert np.array_equal(got, ref)


def test_sjf_padding_parity():
    g = np.random.default_rng(31)
    for B, batch in ((1, 1), (7, 3), (1000, 16), (65536, 32)):
        y = g.integers(1, 20000, size=B).astype(np.int32)
        yhat = y * np.exp(g.normal(0.0, 0.5, size=B))
        order = np.argsort(yhat, kind="stable").astype(np.int32)
        for o in (None, order):
            got = host(estp.sjf_padding(dev(y), None if o is None else dev(o), batch))
            ref = oracle.sjf_padding(y, o, batch)
            assert tuple(int(x) for x in got) == ref
