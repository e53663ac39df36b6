"""ctypes binding of libestp (the C ABI in include/estp.h).

Argument marshalling only: shapes and strides are read from torch tensors,
outputs and workspaces are allocated with torch on the tensors' device, and
every step of the computation runs in the library's HIP kernels on the
given stream (default: the current torch stream).  Tensors a wrapper
allocates are allocated on that same stream, so torch's caching allocator
never hands their memory to other work while the kernels still use it.
There is no fallback: if the library is missing or a call fails, an
exception is raised.
"""
from __future__ import annotations

import contextlib
import ctypes
import math
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("ESTP_LIBRARY") or os.path.join(_HERE, "libestp.so")

ESTP_OK, ESTP_ERR_INVALID_ARG, ESTP_ERR_UNSUPPORTED, ESTP_ERR_WORKSPACE, ESTP_ERR_HIP = range(5)
ESTP_BF16, ESTP_F32 = 0, 1
ESTP_IMPORTANCE_EXCLUDE_SELF = 1
ESTP_NOALLOC_SCRATCH_BYTES = 32 << 20
NORMS = {"none": 0, "zscore": 1, "minmax": 2}
ACTS = {"relu": 0, "gelu_tanh": 1}

EXPORTS = (
    "estp_version", "estp_status_string", "estp_last_error", "estp_debug_checks",
    "estp_token_entropy_workspace_size", "estp_token_entropy", "estp_token_entropy_noalloc",
    "estp_attn_importance_workspace_size", "estp_attn_importance",
    "estp_attn_importance_from_lse_workspace_size", "estp_attn_importance_from_lse",
    "estp_attn_importance_ex_workspace_size", "estp_attn_importance_ex",
    "estp_combine_pool_workspace_size", "estp_combine_pool",
    "estp_predict_workspace_size", "estp_predict",
    "estp_head_train_step_workspace_size", "estp_head_train_step",
    "estp_misalignment", "estp_sjf_padding",
)


class EstpError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status}: {detail}")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_F = ctypes.c_float
_SZ = ctypes.c_size_t
_INT = ctypes.c_int


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libestp.so (built by ``paper_2608_15592_amd.build``) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_15592_amd.build`")
    lib = ctypes.CDLL(path)
    lib.estp_version.restype = _INT
    lib.estp_version.argtypes = []
    lib.estp_status_string.restype = ctypes.c_char_p
    lib.estp_status_string.argtypes = [_INT]
    lib.estp_last_error.restype = ctypes.c_char_p
    lib.estp_last_error.argtypes = []
    lib.estp_debug_checks.restype = _INT
    lib.estp_debug_checks.argtypes = []
    lib.estp_token_entropy_workspace_size.restype = _SZ
    lib.estp_token_entropy_workspace_size.argtypes = [_I64, _I32, _I32, _INT]
    lib.estp_token_entropy.restype = _INT
    lib.estp_token_entropy.argtypes = [_P, _P, _I64, _I32, _I32, _INT, _P, _P, _P, _SZ, _P]
    lib.estp_token_entropy_noalloc.restype = _INT
    lib.estp_token_entropy_noalloc.argtypes = [_P, _P, _I64, _I32, _I32, _INT, _P, _P, _P]
    lib.estp_attn_importance_workspace_size.restype = _SZ
    lib.estp_attn_importance_workspace_size.argtypes = [_I64, _I32, _I32, _I32, _I32, _I32, _I32, _INT]
    lib.estp_attn_importance.restype = _INT
    lib.estp_attn_importance.argtypes = [_P, _P, _P, _I32, _I32, _I64, _I32, _I32, _I32, _I32, _F, _INT, _P, _P,
                                         _SZ, _P]
    lib.estp_attn_importance_from_lse_workspace_size.restype = _SZ
    lib.estp_attn_importance_from_lse_workspace_size.argtypes = [_I64, _I32, _I32, _I32, _I32, _I32, _I32, _INT]
    lib.estp_attn_importance_from_lse.restype = _INT
    lib.estp_attn_importance_from_lse.argtypes = [_P, _P, _P, _P, _I32, _I32, _I64, _I32, _I32, _I32, _I32, _F,
                                                  _INT, _P, _P, _SZ, _P]
    lib.estp_attn_importance_ex_workspace_size.restype = _SZ
    lib.estp_attn_importance_ex_workspace_size.argtypes = [_I64, _I32, _I32, _I32, _I32, _I32, _I32, _INT, _INT]
    lib.estp_attn_importance_ex.restype = _INT
    lib.estp_attn_importance_ex.argtypes = [_P, _P, _P, _P, _I32, _I32, _I64, _I32, _I32, _I32, _I32, _F, _P, _INT,
                                            _INT, _P, _P, _SZ, _P]
    lib.estp_combine_pool_workspace_size.restype = _SZ
    lib.estp_combine_pool_workspace_size.argtypes = [_I64, _I32, _I32, _I32, _INT]
    lib.estp_combine_pool.restype = _INT
    lib.estp_combine_pool.argtypes = [_P, _P, _P, _P, _I32, _I32, _I64, _I32, _F, _F, _F, _INT, _INT, _P, _P, _P,
                                      _P, _SZ, _P]
    lib.estp_predict_workspace_size.restype = _SZ
    lib.estp_predict_workspace_size.argtypes = [_I32, _I32, _I32, _I32]
    lib.estp_predict.restype = _INT
    lib.estp_predict.argtypes = [_P, _I32, _I32, _P, _P, _I32, _INT, _P, _P, _I32, _P, _P, _P, _P, _P, _SZ, _P]
    lib.estp_head_train_step_workspace_size.restype = _SZ
    lib.estp_head_train_step_workspace_size.argtypes = [_I32, _I32, _I32, _I32]
    lib.estp_head_train_step.restype = _INT
    lib.estp_head_train_step.argtypes = [_P, _P, _I32, _I32, _I32, _I32, _INT, _P, _P, _P, _P, _P, _I32, _F, _F, _F,
                                         _F, _F, _F, _P, _P, _SZ, _P]
    lib.estp_misalignment.restype = _INT
    lib.estp_misalignment.argtypes = [_P, _P, _P, _I32, _F, _F, _P, _P]
    lib.estp_sjf_padding.restype = _INT
    lib.estp_sjf_padding.argtypes = [_P, _P, _I32, _I32, _P, _P]
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != ESTP_OK:
        lib = load()
        raise EstpError(status, where, lib.estp_last_error().decode())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return ESTP_BF16
    if t.dtype == torch.float32:
        return ESTP_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


@contextlib.contextmanager
def _on(stream, device):
    """Make ``device`` current and ``stream`` (default: the device's current stream) the
    current stream; yields the stream handle to pass to the library.  Every tensor a
    wrapper allocates inside (outputs, workspace) then belongs to the stream the kernels
    are enqueued on: when it is freed, the caching allocator reuses the block only for
    work ordered after that stream's kernels."""
    with torch.cuda.device(device):
        s = torch.cuda.current_stream(device) if stream is None else stream
        with torch.cuda.stream(s):
            yield ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, name: str, device=None, dtype=None, ndim=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {t.dim()}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _sized(t: torch.Tensor, name: str, n: int, device=None, dtype=None):
    """A device tensor of exactly n elements (contiguous, on ``device``, of ``dtype``)."""
    _need(t, name, device=device, dtype=dtype)
    if t.numel() != n:
        raise ValueError(f"{name} must hold {n} elements, got {t.numel()}")


def _workspace(nbytes: int, device, workspace: Optional[torch.Tensor]):
    if workspace is not None:
        _need(workspace, "workspace", device=device)
    if nbytes == 0:
        return workspace, 0
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return workspace, workspace.numel() * workspace.element_size()


# ----------------------------------------------------------------------------- calls

def token_entropy_workspace_size(n_tok: int, d: int, V: int, dtype=torch.bfloat16) -> int:
    return load().estp_token_entropy_workspace_size(n_tok, d, V, ESTP_BF16 if dtype == torch.bfloat16 else ESTP_F32)


def token_entropy(X: torch.Tensor, W: torch.Tensor, H: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None, stream=None,
                  vocab_argmax: Optional[torch.Tensor] = None) -> torch.Tensor:
    """H[i] = entropy (nats) of softmax(W @ X[i]) over the vocabulary (Eq. 2).

    ``vocab_argmax`` (optional int32 [n_tok] device tensor) is filled with each row's
    most probable next token: the index of its largest logit, lowest index among ties.
    """
    lib = load()
    _need(X, "X", ndim=2)
    _need(W, "W", device=X.device, dtype=X.dtype, ndim=2)
    n_tok, d = X.shape
    V = W.shape[0]
    if W.shape[1] != d:
        raise ValueError("X and W disagree on d")
    if vocab_argmax is not None:
        _sized(vocab_argmax, "vocab_argmax", n_tok, device=X.device, dtype=torch.int32)
    dt = _dtype_code(X)
    with _on(stream, X.device) as st:
        if H is None:
            H = torch.empty(n_tok, dtype=torch.float32, device=X.device)
        _sized(H, "H", n_tok, device=X.device, dtype=torch.float32)
        workspace, wsb = _workspace(lib.estp_token_entropy_workspace_size(n_tok, d, V, dt), X.device, workspace)
        _check(lib.estp_token_entropy(_ptr(X), _ptr(W), n_tok, d, V, dt, _ptr(H), _ptr(vocab_argmax),
                                      _ptr(workspace), wsb, st), "estp_token_entropy")
    return H


def token_entropy_noalloc(X: torch.Tensor, W: torch.Tensor, H: torch.Tensor,
                          vocab_argmax: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """``token_entropy`` through estp_token_entropy_noalloc: the library's own per-GPU scratch
    instead of a workspace, so the call allocates nothing (H and the optional ``vocab_argmax``
    are the caller's).  Calls that overlap on one GPU race on that scratch."""
    lib = load()
    _need(X, "X", ndim=2)
    _need(W, "W", device=X.device, dtype=X.dtype, ndim=2)
    n_tok, d = X.shape
    V = W.shape[0]
    if W.shape[1] != d:
        raise ValueError("X and W disagree on d")
    _sized(H, "H", n_tok, device=X.device, dtype=torch.float32)
    if vocab_argmax is not None:
        _sized(vocab_argmax, "vocab_argmax", n_tok, device=X.device, dtype=torch.int32)
    with _on(stream, X.device) as st:
        _check(lib.estp_token_entropy_noalloc(_ptr(X), _ptr(W), n_tok, d, V, _dtype_code(X), _ptr(H),
                                              _ptr(vocab_argmax), st), "estp_token_entropy_noalloc")
    return H


def _qk_shapes(Q: torch.Tensor, K: torch.Tensor, cu_seqlens: torch.Tensor):
    if Q.dim() == 3:
        Q, K = Q.unsqueeze(0), K.unsqueeze(0)
    _need(Q, "Q", ndim=4)
    _need(K, "K", device=Q.device, dtype=Q.dtype, ndim=4)
    _need(cu_seqlens, "cu_seqlens", device=Q.device, dtype=torch.int32, ndim=1)
    L, n_tok, Hq, dh = Q.shape
    if K.shape[0] != L or K.shape[1] != n_tok or K.shape[3] != dh:
        raise ValueError("Q and K shapes disagree")
    return Q, K, L, n_tok, Hq, K.shape[2], dh


def attn_importance(Q: torch.Tensor, K: torch.Tensor, cu_seqlens: torch.Tensor, max_seqlen: int,
                    scale: Optional[float] = None, S: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """S[j] = column mean of the head-averaged causal attention, summed over layers (Eq. 1).

    Q [L, n_tok, Hq, dh], K [L, n_tok, Hkv, dh] (3-D tensors are one layer).
    """
    lib = load()
    Q, K, L, n_tok, Hq, Hkv, dh = _qk_shapes(Q, K, cu_seqlens)
    B = cu_seqlens.numel() - 1
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    dt = _dtype_code(Q)
    with _on(stream, Q.device) as st:
        if S is None:
            S = torch.empty(n_tok, dtype=torch.float32, device=Q.device)
        _sized(S, "S", n_tok, device=Q.device, dtype=torch.float32)
        ws = lib.estp_attn_importance_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dt)
        workspace, wsb = _workspace(ws, Q.device, workspace)
        _check(lib.estp_attn_importance(_ptr(Q), _ptr(K), _ptr(cu_seqlens), B, int(max_seqlen), n_tok, L, Hq, Hkv, dh,
                                        float(scale), dt, _ptr(S), _ptr(workspace), wsb, st),
               "estp_attn_importance")
    return S


def attn_importance_from_lse(Q: torch.Tensor, K: torch.Tensor, lse: torch.Tensor, cu_seqlens: torch.Tensor,
                             max_seqlen: int, scale: Optional[float] = None, S: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Eq. 1 importance from given per-row natural-log normalisers ``lse`` [L, Hq, n_tok] (a prefill's LSE).

    Q [L, n_tok, Hq, dh], K [L, n_tok, Hkv, dh] (3-D tensors and a 2-D ``lse`` are one layer).
    """
    lib = load()
    Q, K, L, n_tok, Hq, Hkv, dh = _qk_shapes(Q, K, cu_seqlens)
    if lse.dim() == 2:
        lse = lse.unsqueeze(0)
    _need(lse, "lse", device=Q.device, dtype=torch.float32, ndim=3)
    if tuple(lse.shape) != (L, Hq, n_tok):
        raise ValueError(f"lse must be [L, Hq, n_tok] = {(L, Hq, n_tok)}, got {tuple(lse.shape)}")
    B = cu_seqlens.numel() - 1
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    dt = _dtype_code(Q)
    with _on(stream, Q.device) as st:
        if S is None:
            S = torch.empty(n_tok, dtype=torch.float32, device=Q.device)
        _sized(S, "S", n_tok, device=Q.device, dtype=torch.float32)
        ws = lib.estp_attn_importance_from_lse_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dt)
        workspace, wsb = _workspace(ws, Q.device, workspace)
        _check(lib.estp_attn_importance_from_lse(_ptr(Q), _ptr(K), _ptr(lse), _ptr(cu_seqlens), B, int(max_seqlen),
                                                 n_tok, L, Hq, Hkv, dh, float(scale), dt, _ptr(S), _ptr(workspace),
                                                 wsb, st),
               "estp_attn_importance_from_lse")
    return S


def attn_importance_ex(Q: torch.Tensor, K: torch.Tensor, cu_seqlens: torch.Tensor, max_seqlen: int,
                       lse: Optional[torch.Tensor] = None, layer_weights=None, exclude_self: bool = False,
                       scale: Optional[float] = None, S: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Eq. 1 importance with the variants of estp_attn_importance_ex: optional prefill row LSEs
    ``lse`` [L, Hq, n_tok], per-layer weights (host sequence of L floats), and the diagonal
    left out of the column sums (``exclude_self``)."""
    lib = load()
    Q, K, L, n_tok, Hq, Hkv, dh = _qk_shapes(Q, K, cu_seqlens)
    if lse is not None:
        if lse.dim() == 2:
            lse = lse.unsqueeze(0)
        _need(lse, "lse", device=Q.device, dtype=torch.float32, ndim=3)
        if tuple(lse.shape) != (L, Hq, n_tok):
            raise ValueError(f"lse must be [L, Hq, n_tok] = {(L, Hq, n_tok)}")
    lw = None
    if layer_weights is not None:
        if len(layer_weights) != L:
            raise ValueError(f"layer_weights must hold L = {L} values")
        lw = (ctypes.c_float * L)(*[float(x) for x in layer_weights])
    B = cu_seqlens.numel() - 1
    if scale is None:
        scale = 1.0 / math.sqrt(dh)
    dt = _dtype_code(Q)
    flags = ESTP_IMPORTANCE_EXCLUDE_SELF if exclude_self else 0
    with _on(stream, Q.device) as st:
        if S is None:
            S = torch.empty(n_tok, dtype=torch.float32, device=Q.device)
        _sized(S, "S", n_tok, device=Q.device, dtype=torch.float32)
        ws = lib.estp_attn_importance_ex_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dt,
                                                        int(lse is not None))
        workspace, wsb = _workspace(ws, Q.device, workspace)
        _check(lib.estp_attn_importance_ex(_ptr(Q), _ptr(K), _ptr(lse), _ptr(cu_seqlens), B, int(max_seqlen), n_tok, L,
                                           Hq, Hkv, dh, float(scale), lw, flags, dt, _ptr(S), _ptr(workspace), wsb,
                                           st),
               "estp_attn_importance_ex")
    return S


def combine_pool(X: torch.Tensor, S: torch.Tensor, H: torch.Tensor, cu_seqlens: torch.Tensor, max_seqlen: int,
                 lambda1: float, lambda2: float, alpha: float = 1.0, norm: str = "none",
                 pooled: Optional[torch.Tensor] = None, e: Optional[torch.Tensor] = None,
                 top: Optional[torch.Tensor] = None, want_e: bool = True, want_top: bool = True,
                 workspace: Optional[torch.Tensor] = None, stream=None):
    """e = softmax over each prompt of (lambda1 S + lambda2 H) / alpha; pooled[b] = sum e_i X_i (Eq. 3-5).

    Returns ``(pooled [B, d], e [n_tok] or None, top [B] or None)``.
    """
    lib = load()
    _need(X, "X", ndim=2)
    n_tok, d = X.shape
    _sized(S, "S", n_tok, device=X.device, dtype=torch.float32)
    _sized(H, "H", n_tok, device=X.device, dtype=torch.float32)
    _need(cu_seqlens, "cu_seqlens", device=X.device, dtype=torch.int32, ndim=1)
    B = cu_seqlens.numel() - 1
    dt = _dtype_code(X)
    with _on(stream, X.device) as st:
        if pooled is None:
            pooled = torch.empty(B, d, dtype=torch.float32, device=X.device)
        _sized(pooled, "pooled", B * d, device=X.device, dtype=torch.float32)
        if e is None and want_e:
            e = torch.empty(n_tok, dtype=torch.float32, device=X.device)
        if e is not None:
            _sized(e, "e", n_tok, device=X.device, dtype=torch.float32)
        if top is None and want_top:
            top = torch.empty(B, dtype=torch.int32, device=X.device)
        if top is not None:
            _sized(top, "top", B, device=X.device, dtype=torch.int32)
        workspace, wsb = _workspace(lib.estp_combine_pool_workspace_size(n_tok, B, max_seqlen, d, dt), X.device,
                                    workspace)
        _check(lib.estp_combine_pool(_ptr(X), _ptr(S), _ptr(H), _ptr(cu_seqlens), B, int(max_seqlen), n_tok, d,
                                     float(lambda1), float(lambda2), float(alpha), NORMS[norm], dt, _ptr(pooled),
                                     _ptr(e), _ptr(top), _ptr(workspace), wsb, st),
               "estp_combine_pool")
    return pooled, e, top


def predict(pooled: torch.Tensor, W1: torch.Tensor, b1: Optional[torch.Tensor], W2: torch.Tensor,
            b2: Optional[torch.Tensor], centres: Optional[torch.Tensor] = None, act: str = "relu",
            want_order: bool = True, workspace: Optional[torch.Tensor] = None, stream=None):
    """Length head: returns ``(yhat [B], bin [B] or None, order [B] or None)`` (Section 4.3, Eq. 7)."""
    lib = load()
    _need(pooled, "pooled", dtype=torch.float32, ndim=2)
    for t, n in ((W1, "W1"), (W2, "W2")):
        _need(t, n, device=pooled.device, dtype=torch.float32, ndim=2)
    B, d = pooled.shape
    Hd, K = W1.shape[0], W2.shape[0]
    if W1.shape[1] != d or W2.shape[1] != Hd:
        raise ValueError("head weight shapes disagree")
    for t, n, size in ((b1, "b1", Hd), (b2, "b2", K), (centres, "centres", K)):
        if t is not None:
            _sized(t, n, size, device=pooled.device, dtype=torch.float32)
    with _on(stream, pooled.device) as st:
        yhat = torch.empty(B, dtype=torch.float32, device=pooled.device)
        bins = torch.empty(B, dtype=torch.int32, device=pooled.device) if K > 1 else None
        order = torch.empty(B, dtype=torch.int32, device=pooled.device) if want_order else None
        workspace, wsb = _workspace(lib.estp_predict_workspace_size(B, d, Hd, K), pooled.device, workspace)
        _check(lib.estp_predict(_ptr(pooled), B, d, _ptr(W1), _ptr(b1), Hd, ACTS[act], _ptr(W2), _ptr(b2), K,
                                _ptr(centres), _ptr(yhat), _ptr(bins), _ptr(order), _ptr(workspace), wsb, st),
               "estp_predict")
    return yhat, bins, order


def head_param_views(theta: torch.Tensor, d: int, hidden: int, K: int):
    """(W1, b1, W2, b2) views into a flat parameter vector laid out as estp_head_train_step expects."""
    n1 = hidden * d
    W1 = theta[:n1].view(hidden, d)
    b1 = theta[n1:n1 + hidden]
    W2 = theta[n1 + hidden:n1 + hidden + K * hidden].view(K, hidden)
    b2 = theta[n1 + hidden + K * hidden:n1 + hidden + K * hidden + K]
    return W1, b1, W2, b2


def head_train_step(pooled: torch.Tensor, y: torch.Tensor, edges: torch.Tensor, centres: torch.Tensor,
                    theta: torch.Tensor, m: torch.Tensor, v: torch.Tensor, hidden: int, step: int,
                    lambda3: float, lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                    weight_decay: float = 0.01, act: str = "relu", loss: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """One Eq. 8 / AdamW step of the K-bin length head; updates ``theta``, ``m``, ``v`` in place and
    returns the batch loss (a 1-element device tensor) computed before the update."""
    lib = load()
    _need(pooled, "pooled", dtype=torch.float32, ndim=2)
    dev_ = pooled.device
    for t, n in ((y, "y"), (edges, "edges"), (centres, "centres"), (theta, "theta"), (m, "m"), (v, "v")):
        _need(t, n, device=dev_, dtype=torch.float32, ndim=1)
    B, d = pooled.shape
    K = centres.numel()
    if edges.numel() != K + 1 or y.numel() != B:
        raise ValueError("edges must hold K+1 values and y B values")
    n = hidden * d + hidden + K * hidden + K
    if theta.numel() != n or m.numel() != n or v.numel() != n:
        raise ValueError(f"theta, m, v must hold {n} values")
    with _on(stream, dev_) as st:
        if loss is None:
            loss = torch.empty(1, dtype=torch.float32, device=dev_)
        _sized(loss, "loss", 1, device=dev_, dtype=torch.float32)
        workspace, wsb = _workspace(lib.estp_head_train_step_workspace_size(B, d, hidden, K), dev_, workspace)
        _check(lib.estp_head_train_step(_ptr(pooled), _ptr(y), B, d, hidden, K, ACTS[act], _ptr(edges), _ptr(centres),
                                        _ptr(theta), _ptr(m), _ptr(v), int(step), float(lambda3), float(lr),
                                        float(beta1), float(beta2), float(eps), float(weight_decay), _ptr(loss),
                                        _ptr(workspace), wsb, st),
               "estp_head_train_step")
    return loss


def misalignment(H: torch.Tensor, S: torch.Tensor, cu_seqlens: torch.Tensor, frac_low: float = 0.4,
                 frac_high: float = 0.4, stream=None) -> torch.Tensor:
    """Per-prompt counts [B, 4] of the entropy / semantics rank split (Fig. 1b): #high-H,
    #high-H that are low-S, #low-H, #low-H that are high-S."""
    lib = load()
    _need(H, "H", dtype=torch.float32, ndim=1)
    _sized(S, "S", H.numel(), device=H.device, dtype=torch.float32)
    _need(cu_seqlens, "cu_seqlens", device=H.device, dtype=torch.int32, ndim=1)
    B = cu_seqlens.numel() - 1
    with _on(stream, H.device) as st:
        counts = torch.empty(B, 4, dtype=torch.int32, device=H.device)
        _check(lib.estp_misalignment(_ptr(H), _ptr(S), _ptr(cu_seqlens), B, float(frac_low), float(frac_high),
                                     _ptr(counts), st), "estp_misalignment")
    return counts


def sjf_padding(lengths: torch.Tensor, order: Optional[torch.Tensor], batch: int, stream=None) -> torch.Tensor:
    """(padded tokens, useful tokens, sum of completion times) of static batches taken in ``order``."""
    lib = load()
    _need(lengths, "lengths", dtype=torch.int32, ndim=1)
    if order is not None:
        _sized(order, "order", lengths.numel(), device=lengths.device, dtype=torch.int32)
    with _on(stream, lengths.device) as st:
        out = torch.empty(3, dtype=torch.int64, device=lengths.device)
        _check(lib.estp_sjf_padding(_ptr(lengths), _ptr(order), lengths.numel(), int(batch), _ptr(out), st),
               "estp_sjf_padding")
    return out
