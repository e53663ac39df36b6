"""Sizes past the 32-bit boundaries, through the C ABI.

X [n_tok, 4096] and Q [1, n_tok, 32, 128] hold 2.21e9 elements each (4.42 GB in bf16), so byte
offsets into X pass 2^32 and element offsets into Q pass 2^31 at token 524288; prompt 256 straddles
that token.  The checked prompts (first, straddling, last) and sampled entropy rows around the
boundary are compared with the oracle; every other prompt with properties that hold at any size.

The big tensors are built on the device from synthetic base blocks of 8192 rows by an exact
row-dependent transform: row i is base row i mod 8192 rotated by 8 (i // 8192) features.  Rows
8192 apart therefore still differ, so a read at a wrong offset changes the result.  The host
rebuilds the rows it checks with the same transform.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15592_amd as estp
import synth
from synth import inputs as I
from tests._util import check_argmax_margin, dev, host, rel_l2

pytestmark = pytest.mark.gpu

BASE = 8192
LENGTHS = np.array([1024] + [2048] * 263)  # 539,648 tokens; prompt 256 spans tokens 523264..525311
BOUNDARY = 1 << 19                          # token whose X byte offset is 2^32 (d = 4096, bf16)
D, V, HQ, HKV, DH = 4096, 512, 32, 8, 128


def _expand(base: torch.Tensor, n: int) -> torch.Tensor:
    out = torch.empty((n, base.shape[1]), dtype=base.dtype, device=base.device)
    for k in range(math.ceil(n / BASE)):
        lo, hi = k * BASE, min(n, (k + 1) * BASE)
        out[lo:hi] = torch.roll(base[: hi - lo], shifts=8 * k, dims=1)
    return out


def _rows(base: np.ndarray, rows) -> np.ndarray:
    return np.stack([np.roll(base[i % BASE], 8 * (i // BASE)) for i in rows])


@pytest.fixture(scope="module")
def big():
    w = synth.get_workload("llama", V=V, L=1)
    one = np.array([BASE])
    xb = I.hidden_rows(w, 11, lengths=one)                       # [8192, 4096] bf16 bits
    qb = I.qk_layer(w, "q", 0, 12, lengths=one).reshape(BASE, HQ * DH)
    kb = I.qk_layer(w, "k", 0, 13, lengths=one).reshape(BASE, HKV * DH)
    W = I.lm_head_rows(w, 14)                                    # [512, 4096]
    n = int(LENGTHS.sum())
    assert n * D > (1 << 31) and n * HQ * DH > (1 << 31)
    cu = I.cu_seqlens_from_lengths(LENGTHS)
    g = np.random.default_rng(15)
    S = (g.random(n) / 2048).astype(np.float32)
    H = (g.random(n) * 6).astype(np.float32)
    yield {"xb": xb, "qb": qb, "kb": kb, "W": W, "cu": cu, "S": S, "H": H, "n": n}
    torch.cuda.empty_cache()


def test_entropy_past_4gib(big):
    n = big["n"]
    X = _expand(dev(big["xb"]), n)
    Hd = host(estp.token_entropy(X, dev(big["W"])))
    del X
    torch.cuda.empty_cache()
    g = np.random.default_rng(0)
    rows = sorted(set([0, BASE - 1, BASE, BOUNDARY - 1, BOUNDARY, BOUNDARY + 1, BOUNDARY + BASE, n - 1])
                  | set(g.choice(n, size=24, replace=False).tolist()))
    ref = oracle.token_entropy(_rows(big["xb"], rows), big["W"])
    err = np.abs(Hd[rows] - ref).max()
    print(f"entropy at {n} tokens: max |dH| over {len(rows)} rows = {err:.2e}")
    assert err <= 2e-3
    assert np.all(Hd >= 0) and np.all(Hd <= np.log(V) + 2e-3)


# The pooling kernel a call takes follows from the batch and the stated max_seqlen: prompts within 12.5%
# of max_seqlen that fill the chip take the whole-prompt kernel, other batches of prompts up to 8192
# tokens the length-sized-slice kernel, and a max_seqlen above 8192 the chunked pair.  Prompt 256
# straddles token 2^19, where X's byte offset passes 2^32.
@pytest.mark.parametrize("max_seqlen", [2048, 4096, 9000], ids=["whole-prompt-kernel", "ragged-kernel", "chunked"])
def test_combine_pool_past_4gib(big, max_seqlen):
    lengths, cu, n = LENGTHS, big["cu"], big["n"]
    X = _expand(dev(big["xb"]), n)
    pooled, e, top = estp.combine_pool(X, dev(big["S"]), dev(big["H"]), dev(cu), max_seqlen, 0.5, 0.5, 1.0, "none")
    pooled, e, top = host(pooled), host(e), host(top)
    del X
    torch.cuda.empty_cache()
    B = len(lengths)
    for b in (0, 256, B - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        cu_b = np.array([0, hi - lo])
        eb, tb = oracle.combine_weights(big["S"][lo:hi], big["H"][lo:hi], cu_b, 0.5, 0.5, 1.0, "none")
        pb = oracle.pool(_rows(big["xb"], range(lo, hi)), eb, cu_b)[0]
        assert rel_l2(pooled[b], pb) <= 1e-3, b
        np.testing.assert_allclose(e[lo:hi], eb, rtol=1e-4, atol=1e-9)
        check_argmax_margin(int(top[b]) - lo, eb, 1e-6 * eb.max())
    sums = np.add.reduceat(e.astype(np.float64), cu[:-1].astype(np.int64))
    np.testing.assert_allclose(sums, 1.0, atol=1e-4)


def test_importance_past_2g_elements(big):
    n, cu = big["n"], big["cu"]
    Q = _expand(dev(big["qb"]), n).view(1, n, HQ, DH)
    K = _expand(dev(big["kb"]), n).view(1, n, HKV, DH)
    S = host(estp.attn_importance(Q, K, dev(cu), int(LENGTHS.max())))
    del Q, K
    torch.cuda.empty_cache()
    B = len(LENGTHS)
    for b in (0, 256, B - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        q = _rows(big["qb"], range(lo, hi)).reshape(1, hi - lo, HQ, DH)
        k = _rows(big["kb"], range(lo, hi)).reshape(1, hi - lo, HKV, DH)
        ref = oracle.attn_importance(q, k, np.array([0, hi - lo]))
        rel = np.abs(S[lo:hi] - ref) / ref
        print(f"prompt {b} (tokens {lo}..{hi - 1}): max rel |dS| = {rel.max():.2e}")
        assert np.all(np.abs(S[lo:hi] - ref) <= 1e-3 * ref + 1e-12), b
    sums = np.add.reduceat(S.astype(np.float64), cu[:-1].astype(np.int64))
    np.testing.assert_allclose(sums, 1.0, atol=1e-4)
