"""estp_token_entropy_noalloc (the library's own per-GPU scratch, no workspace, no allocation)
against estp_token_entropy (caller workspace), through the C ABI.

Both run the same kernels, so H and the most probable next token must agree bit for bit; the
second call of each pair is smaller than the first (the scratch keeps the previous call's
contents, which must not leak into a smaller call).  The smaller inputs are also checked
against the fp64 oracle (|dH| <= 2e-3 nats, argmax under the margin rule).  A shape whose
partial states exceed the scratch is refused on the host.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15592_amd as estp
from paper_2608_15592_amd import _lib
from synth import inputs as I
from tests._util import check_vocab_argmax, dev, host

pytestmark = pytest.mark.gpu


def _inputs(n, d, V, seed, f32):
    g = np.random.default_rng(seed)
    X = g.standard_normal((n, d)).astype(np.float32)
    X /= np.sqrt((X * X).mean(axis=1, keepdims=True))
    W = (g.standard_normal((V, d)) * 0.02).astype(np.float32)
    if not f32:
        X, W = I.f32_to_bf16_bits(X), I.f32_to_bf16_bits(W)
    return X, W


def _noalloc(lib, Xd, Wd, H, am):
    n, d = Xd.shape
    rc = lib.estp_token_entropy_noalloc(ctypes.c_void_p(Xd.data_ptr()), ctypes.c_void_p(Wd.data_ptr()), n, d,
                                        Wd.shape[0], _lib.ESTP_F32 if Xd.dtype == torch.float32 else _lib.ESTP_BF16,
                                        ctypes.c_void_p(H.data_ptr()), ctypes.c_void_p(am.data_ptr()),
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, lib.estp_last_error()


@pytest.mark.parametrize("f32", [False, True], ids=["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(f32):
    lib = estp.load()
    # (n_tok, d, V): a large call, then a smaller one on the same scratch
    for n, d, V, seed in ((20000, 1024, 40000, 11), (700, 256, 5000, 12)):
        print(f"noalloc {'f32' if f32 else 'bf16'}: n_tok={n} d={d} V={V}", flush=True)
        X, W = _inputs(n, d, V, seed, f32)
        Xd, Wd = dev(X), dev(W)
        am_ref = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        H_ref = estp.token_entropy(Xd, Wd, vocab_argmax=am_ref)
        H = torch.full((n,), float("nan"), device="cuda")
        am = torch.full((n,), -2, dtype=torch.int32, device="cuda")
        _noalloc(lib, Xd, Wd, H, am)
        torch.cuda.synchronize()
        assert torch.equal(H, H_ref)
        assert torch.equal(am, am_ref)
    # the smaller call against the oracle
    ref = oracle.token_entropy(X, W)
    assert np.abs(host(H) - ref).max() <= 2e-3
    check_vocab_argmax(host(am), X, W)


def test_noalloc_refuses_shapes_past_the_scratch():
    lib = estp.load()
    d, V = 32, 4096  # 16 vocabulary slices: 320 bytes of partial states per token
    per_tok = 5 * 16 * 4
    n = _lib.ESTP_NOALLOC_SCRATCH_BYTES // per_tok + 1
    assert lib.estp_token_entropy_workspace_size(n, d, V, 0) > _lib.ESTP_NOALLOC_SCRATCH_BYTES
    # real buffers of the claimed size, so nothing could be read out of bounds even if a check slipped
    X = torch.zeros(n, d, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(V, d, dtype=torch.bfloat16, device="cuda")
    H = torch.empty(n, device="cuda")
    with pytest.raises(estp.EstpError) as ei:
        _lib.token_entropy_noalloc(X, W, H)
    assert ei.value.status == _lib.ESTP_ERR_UNSUPPORTED
    assert "scratch" in str(ei.value)
    # a shape just inside the limit is accepted (and exact: zero weights give uniform logits, ln V)
    n_ok = _lib.ESTP_NOALLOC_SCRATCH_BYTES // per_tok - 512
    assert lib.estp_token_entropy_workspace_size(n_ok, d, V, 0) <= _lib.ESTP_NOALLOC_SCRATCH_BYTES
    _lib.token_entropy_noalloc(X[:n_ok], W, H[:n_ok])
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(H[:n_ok]), np.log(V), atol=2e-3)
