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
