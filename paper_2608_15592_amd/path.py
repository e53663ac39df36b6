"""The whole ESTP path on one stream: entropy -> importance -> fusion + pooling -> length head."""
from __future__ import annotations

from typing import Optional

import torch

from . import _lib


def run_path(X: torch.Tensor, W: torch.Tensor, Q: torch.Tensor, K: torch.Tensor, cu_seqlens: torch.Tensor,
             max_seqlen: int, lambda1: float, lambda2: float, alpha: float = 1.0, norm: str = "none",
             head: Optional[tuple] = None, act: str = "relu", scale: Optional[float] = None,
             bufs: Optional[dict] = None, stream=None) -> dict:
    """Run the four library calls back to back on ``stream`` (default: current).

    ``head`` is ``(W1, b1, W2, b2, centres)``.  ``bufs`` (optional) holds
    preallocated outputs and workspaces keyed by name so that repeated calls
    allocate nothing: H, S, pooled, e, top, ws_entropy, ws_importance, ws_pool,
    ws_predict; an int32 [n_tok] ``vocab_argmax`` entry, when present, also
    receives each token's most probable next token.
    """
    b = bufs if bufs is not None else {}
    H = _lib.token_entropy(X, W, H=b.get("H"), workspace=b.get("ws_entropy"), stream=stream,
                           vocab_argmax=b.get("vocab_argmax"))
    S = _lib.attn_importance(Q, K, cu_seqlens, max_seqlen, scale=scale, S=b.get("S"),
                             workspace=b.get("ws_importance"), stream=stream)
    pooled, e, top = _lib.combine_pool(X, S, H, cu_seqlens, max_seqlen, lambda1, lambda2, alpha, norm,
                                       pooled=b.get("pooled"), e=b.get("e"), top=b.get("top"),
                                       workspace=b.get("ws_pool"), stream=stream)
    out = {"H": H, "S": S, "pooled": pooled, "e": e, "top": top}
    if b.get("vocab_argmax") is not None:
        out["vocab_argmax"] = b["vocab_argmax"]
    if head is not None:
        W1, b1, W2, b2, centres = head
        out["yhat"], out["bin"], out["order"] = _lib.predict(pooled, W1, b1, W2, b2, centres, act,
                                                             workspace=b.get("ws_predict"), stream=stream)
    return out


def alloc_buffers(n_tok: int, B: int, max_seqlen: int, d: int, V: int, L: int, Hq: int, Hkv: int, dh: int,
                  hidden: int, n_bins: int, device, dtype=torch.bfloat16) -> dict:
    """Outputs and workspaces for ``run_path`` sized for one workload."""
    lib = _lib.load()
    dt = _lib.ESTP_BF16 if dtype == torch.bfloat16 else _lib.ESTP_F32

    def ws(n):
        return torch.empty(max(int(n), 256), dtype=torch.uint8, device=device)

    return {
        "H": torch.empty(n_tok, dtype=torch.float32, device=device),
        "S": torch.empty(n_tok, dtype=torch.float32, device=device),
        "pooled": torch.empty(B, d, dtype=torch.float32, device=device),
        "e": torch.empty(n_tok, dtype=torch.float32, device=device),
        "top": torch.empty(B, dtype=torch.int32, device=device),
        "ws_entropy": ws(lib.estp_token_entropy_workspace_size(n_tok, d, V, dt)),
        "ws_importance": ws(lib.estp_attn_importance_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dt)),
        "ws_pool": ws(lib.estp_combine_pool_workspace_size(n_tok, B, max_seqlen, d, dt)),
        "ws_predict": ws(lib.estp_predict_workspace_size(B, d, hidden, n_bins)),
    }
