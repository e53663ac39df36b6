"""The Python binding refuses mis-sized or misplaced tensors before the library is called, so a
caller's mistake can never become an out-of-bounds device access."""
import pytest
import torch

import paper_2608_15592_amd as estp

pytestmark = pytest.mark.gpu


def _cu(lengths):
    out = [0]
    for n in lengths:
        out.append(out[-1] + n)
    return torch.tensor(out, dtype=torch.int32, device="cuda")


def test_importance_rejects_short_output():
    Q = torch.zeros(1, 40, 2, 32, dtype=torch.bfloat16, device="cuda")
    K = torch.zeros(1, 40, 2, 32, dtype=torch.bfloat16, device="cuda")
    cu = _cu([40])
    short = torch.empty(39, device="cuda")
    with pytest.raises(ValueError, match="S must hold 40"):
        estp.attn_importance(Q, K, cu, 40, S=short)
    lse = torch.zeros(1, 2, 40, device="cuda")
    with pytest.raises(ValueError, match="S must hold 40"):
        estp.attn_importance_from_lse(Q, K, lse, cu, 40, S=short)
    with pytest.raises(ValueError, match="S must hold 40"):
        estp.attn_importance_ex(Q, K, cu, 40, S=short)


def test_combine_pool_rejects_mis_sized_tensors():
    X = torch.zeros(50, 64, dtype=torch.bfloat16, device="cuda")
    S = torch.zeros(50, device="cuda")
    H = torch.zeros(50, device="cuda")
    cu = _cu([20, 30])
    with pytest.raises(ValueError, match="S must hold 50"):
        estp.combine_pool(X, S[:49], H, cu, 30, 0.5, 0.5)
    with pytest.raises(ValueError, match="pooled must hold 128"):
        estp.combine_pool(X, S, H, cu, 30, 0.5, 0.5, pooled=torch.empty(1, 64, device="cuda"))
    with pytest.raises(ValueError, match="e must hold 50"):
        estp.combine_pool(X, S, H, cu, 30, 0.5, 0.5, e=torch.empty(10, device="cuda"))
    with pytest.raises(ValueError, match="top must hold 2"):
        estp.combine_pool(X, S, H, cu, 30, 0.5, 0.5, top=torch.empty(1, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="workspace must be a device tensor"):
        estp.combine_pool(X, S, H, cu, 30, 0.5, 0.5, workspace=torch.empty(1 << 20, dtype=torch.uint8))


def test_predict_rejects_mis_sized_head():
    pooled = torch.zeros(3, 64, device="cuda")
    W1 = torch.zeros(16, 64, device="cuda")
    W2 = torch.zeros(4, 16, device="cuda")
    with pytest.raises(ValueError, match="b1 must hold 16"):
        estp.predict(pooled, W1, torch.zeros(15, device="cuda"), W2, None, torch.arange(4.0, device="cuda"))
    with pytest.raises(ValueError, match="centres must hold 4"):
        estp.predict(pooled, W1, None, W2, None, torch.arange(3.0, device="cuda"))


def test_analyses_reject_mis_sized_inputs():
    H = torch.zeros(30, device="cuda")
    with pytest.raises(ValueError, match="S must hold 30"):
        estp.misalignment(H, torch.zeros(29, device="cuda"), _cu([30]))
    lengths = torch.ones(10, dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError, match="order must hold 10"):
        estp.sjf_padding(lengths, torch.arange(9, dtype=torch.int32, device="cuda"), 4)


def test_side_stream_internal_workspace_is_not_reused_early():
    # A call on a side stream with no workspace: the binding allocates workspace and outputs on
    # that stream, so memory allocated and overwritten on the default stream right after the
    # call returns can never land in blocks the side stream's kernels still use.
    g = torch.Generator(device="cuda").manual_seed(3)
    n, L, Hq, Hkv, dh = 4096, 2, 16, 4, 128
    Q = torch.randn(L, n, Hq, dh, device="cuda", generator=g).to(torch.bfloat16)
    K = torch.randn(L, n, Hkv, dh, device="cuda", generator=g).to(torch.bfloat16)
    cu = _cu([2048, 1024, 1024])
    X = torch.randn(n, 1024, device="cuda", generator=g).to(torch.bfloat16)
    W = (0.02 * torch.randn(8192, 1024, device="cuda", generator=g)).to(torch.bfloat16)
    ref_S = estp.attn_importance(Q, K, cu, 2048).clone()
    ref_H = estp.token_entropy(X, W).clone()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    for _ in range(3):
        side.wait_stream(torch.cuda.current_stream())
        S = estp.attn_importance(Q, K, cu, 2048, stream=side)
        H = estp.token_entropy(X, W, stream=side)
        # immediately claim and scribble over memory on the default stream
        junk = [torch.full((1 << 22,), float("nan"), device="cuda") for _ in range(8)]
        side.synchronize()
        torch.cuda.synchronize()
        assert torch.equal(S, ref_S)
        assert torch.equal(H, ref_H)
        del junk, S, H
