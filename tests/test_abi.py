"""The C ABI library: it loads, exports every symbol include/estp.h declares, and rejects
invalid arguments on the host before any device work."""
import ctypes
import os
import re

import pytest

import paper_2608_15592_amd as estp
from paper_2608_15592_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "estp.h")


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"ESTP_API\s+[\w\s\*]+?\b(estp_\w+)\s*\(", txt)))


def test_header_declares_expected_calls():
    names = _declared()
    for n in ("estp_token_entropy", "estp_attn_importance", "estp_combine_pool", "estp_predict"):
        assert n in names
    assert set(names) == set(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = estp.load()
    for n in _declared():
        assert hasattr(lib, n), n
    header = open(os.path.join(ROOT, "include", "estp.h")).read()
    assert lib.estp_version() == int(re.search(r"#define ESTP_VERSION (\d+)", header).group(1))
    for code in range(5):
        assert lib.estp_status_string(code).startswith(b"ESTP_")


def _gpu_present():
    import torch
    return torch.cuda.is_available()


# Every case below fails host-side validation; they run only where no GPU is visible, so
# that the fake (aligned, non-null) pointers can never reach a kernel.
needs_no_gpu = pytest.mark.skipif(_gpu_present(), reason="host-validation cases use fake pointers")

FAKE = ctypes.c_void_p(1 << 20)
UNALIGNED = ctypes.c_void_p((1 << 20) + 2)
WS = ctypes.c_void_p(1 << 24)


@needs_no_gpu
def test_entropy_validation():
    lib = estp.load()
    ws = lib.estp_token_entropy_workspace_size(100, 64, 1000, 0)
    assert ws > 0
    cases = [
        ((None, FAKE, 100, 64, 1000, 0, FAKE, None, WS, ws, None), 1),        # null X
        ((FAKE, FAKE, 0, 64, 1000, 0, FAKE, None, WS, ws, None), 1),          # n_tok < 1
        ((FAKE, FAKE, 100, 60, 1000, 0, FAKE, None, WS, ws, None), 1),        # d % 8
        ((FAKE, FAKE, 100, 64, 0, 0, FAKE, None, WS, ws, None), 1),           # V < 1
        ((FAKE, FAKE, 100, 64, 1000, 7, FAKE, None, WS, ws, None), 1),        # unknown dtype
        ((FAKE, FAKE, 100, 40, 1000, 0, FAKE, None, WS, ws, None), 2),        # bf16: d not a multiple of 32
        ((FAKE, FAKE, 100, 40, 1000, 1, FAKE, None, WS, ws - 1, None), 3),    # f32 takes any d % 8 == 0
        ((UNALIGNED, FAKE, 100, 64, 1000, 0, FAKE, None, WS, ws, None), 1),   # alignment
        ((FAKE, FAKE, 100, 64, 1000, 0, FAKE, UNALIGNED, WS, ws, None), 1),   # argmax output alignment
        ((FAKE, FAKE, 100, 64, 1000, 0, FAKE, None, WS, ws - 1, None), 3),    # workspace short
        ((FAKE, FAKE, 100, 64, 1000, 0, FAKE, None, None, ws, None), 1),      # workspace null
    ]
    for args, code in cases:
        assert lib.estp_token_entropy(*args) == code, (args, lib.estp_last_error())
        assert lib.estp_last_error()


@needs_no_gpu
def test_entropy_noalloc_validation():
    # the no-allocation variant refuses, on the host, the same invalid arguments and every shape
    # whose partial states exceed the library's scratch (its size is in the header)
    lib = estp.load()
    limit = _lib.ESTP_NOALLOC_SCRATCH_BYTES
    assert re.search(r"#define ESTP_NOALLOC_SCRATCH_BYTES \(32u << 20\)", open(HEADER).read())
    assert limit == 32 << 20
    n_big = limit // (5 * 16 * 4) + 1
    assert lib.estp_token_entropy_workspace_size(n_big, 32, 4096, 0) > limit
    cases = [
        ((None, FAKE, 100, 64, 1000, 0, FAKE, None, None), 1),               # null X
        ((FAKE, FAKE, 100, 60, 1000, 0, FAKE, None, None), 1),               # d % 8
        ((FAKE, FAKE, 100, 40, 1000, 0, FAKE, None, None), 2),               # bf16 d % 32
        ((FAKE, FAKE, 100, 64, 1000, 0, FAKE, UNALIGNED, None), 1),          # argmax alignment
        ((FAKE, FAKE, n_big, 32, 4096, 0, FAKE, None, None), 2),             # past the scratch
        ((FAKE, FAKE, 4 * n_big, 32, 1000, 1, FAKE, FAKE, None), 2),         # fp32, 4 slices, past it
    ]
    for args, code in cases:
        assert lib.estp_token_entropy_noalloc(*args) == code, (args, lib.estp_last_error())
        assert lib.estp_last_error()
    lib.estp_token_entropy_noalloc(FAKE, FAKE, n_big, 32, 4096, 0, FAKE, None, None)
    assert b"scratch" in lib.estp_last_error()


@needs_no_gpu
def test_importance_validation():
    lib = estp.load()
    ws = lib.estp_attn_importance_workspace_size(100, 2, 60, 1, 4, 2, 64, 0)
    base = [FAKE, FAKE, FAKE, 2, 60, 100, 1, 4, 2, 64, 0.125, 0, FAKE, WS, ws, None]

    def call(**kw):
        a = list(base)
        idx = {"Q": 0, "B": 3, "max_seqlen": 4, "n_tok": 5, "L": 6, "Hq": 7, "Hkv": 8, "dh": 9, "scale": 10,
               "dtype": 11, "S": 12, "ws": 13, "wsb": 14}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.estp_attn_importance(*a)

    assert call(Q=None) == 1
    assert call(B=0) == 1
    assert call(Hq=5) == 1                # Hq % Hkv
    assert call(scale=0.0) == 1
    assert call(scale=float("inf")) == 1
    assert call(max_seqlen=101) == 1      # longer than n_tok
    assert call(dh=96) == 2
    assert call(dtype=1, wsb=ws - 1) == 3  # f32 accepted, then the workspace check
    assert call(wsb=ws - 1) == 3
    assert call(Q=UNALIGNED) == 1


@needs_no_gpu
def test_importance_from_lse_validation():
    lib = estp.load()
    ws = lib.estp_attn_importance_from_lse_workspace_size(100, 2, 60, 1, 4, 2, 64, 0)
    assert 0 < ws < lib.estp_attn_importance_workspace_size(100, 2, 60, 1, 4, 2, 64, 0)  # no row-LSE buffer
    base = [FAKE, FAKE, FAKE, FAKE, 2, 60, 100, 1, 4, 2, 64, 0.125, 0, FAKE, WS, ws, None]

    def call(**kw):
        a = list(base)
        idx = {"Q": 0, "lse": 2, "B": 4, "Hq": 8, "dh": 10, "scale": 11, "dtype": 12, "wsb": 15}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.estp_attn_importance_from_lse(*a)

    assert call(Q=None) == 1
    assert call(lse=None) == 1
    assert call(B=0) == 1
    assert call(Hq=5) == 1
    assert call(scale=-1.0) == 1
    assert call(dh=96) == 2
    assert call(dtype=1, wsb=ws - 1) == 3  # f32 accepted, then the workspace check
    assert call(wsb=ws - 1) == 3
    assert call(Q=UNALIGNED) == 1


@needs_no_gpu
def test_combine_pool_validation():
    lib = estp.load()
    ws = lib.estp_combine_pool_workspace_size(100, 2, 60, 64, 0)
    base = [FAKE, FAKE, FAKE, FAKE, 2, 60, 100, 64, 0.5, 0.5, 1.0, 0, 0, FAKE, None, None, WS, ws, None]

    def call(**kw):
        a = list(base)
        idx = {"X": 0, "d": 7, "l1": 8, "alpha": 10, "norm": 11, "dtype": 12, "pooled": 13, "wsb": 17}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.estp_combine_pool(*a)

    assert call(X=None) == 1
    assert call(pooled=None) == 1
    assert call(d=12) == 1
    assert call(alpha=0.0) == 1
    assert call(alpha=-1.0) == 1
    assert call(alpha=float("nan")) == 1
    assert call(l1=float("nan")) == 1
    assert call(norm=5) == 1
    assert call(dtype=3) == 1
    assert call(wsb=ws - 1) == 3


@needs_no_gpu
def test_predict_validation():
    lib = estp.load()
    ws = lib.estp_predict_workspace_size(4, 64, 32, 8)
    base = [FAKE, 4, 64, FAKE, None, 32, 0, FAKE, None, 8, FAKE, FAKE, None, None, WS, ws, None]

    def call(**kw):
        a = list(base)
        idx = {"pooled": 0, "B": 1, "act": 6, "K": 9, "centres": 10, "wsb": 15}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.estp_predict(*a)

    assert call(pooled=None) == 1
    assert call(B=0) == 1
    assert call(B=70000) == 1
    assert call(K=2000) == 1
    assert call(centres=None) == 1      # K > 1 needs centres
    assert call(act=9) == 1
    assert call(wsb=ws - 1) == 3


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError):
        _lib.load.__wrapped__(str(tmp_path / "missing.so")) if hasattr(_lib.load, "__wrapped__") else \
            _load_fresh(str(tmp_path / "missing.so"))


def _load_fresh(path):
    saved = _lib._lib
    try:
        _lib._lib = None
        return _lib.load(path)
    finally:
        _lib._lib = saved


@needs_no_gpu
def test_head_train_step_validation():
    lib = estp.load()
    ws = lib.estp_head_train_step_workspace_size(8, 64, 32, 6)
    assert ws > 0
    base = [FAKE, FAKE, 8, 64, 32, 6, 0, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 0.5, 1e-3, 0.9, 0.999, 1e-8, 0.01, None, WS,
            ws, None]

    def call(**kw):
        a = list(base)
        idx = {"pooled": 0, "B": 2, "d": 3, "K": 5, "act": 6, "theta": 9, "step": 12, "lambda3": 13, "lr": 14,
               "beta1": 15, "eps": 17, "wsb": 21}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.estp_head_train_step(*a)

    assert call(pooled=None) == 1
    assert call(B=0) == 1
    assert call(K=1) == 1                 # Eq. 8 needs bins
    assert call(d=66) == 1                # d % 4
    assert call(act=5) == 1
    assert call(step=0) == 1
    assert call(lambda3=1.5) == 1
    assert call(lr=-1.0) == 1
    assert call(beta1=1.0) == 1
    assert call(eps=0.0) == 1
    assert call(theta=UNALIGNED) == 1
    assert call(wsb=ws - 1) == 3


@needs_no_gpu
def test_importance_ex_validation():
    lib = estp.load()
    ws2 = lib.estp_attn_importance_ex_workspace_size(100, 2, 60, 2, 4, 2, 64, 0, 0)
    ws1 = lib.estp_attn_importance_ex_workspace_size(100, 2, 60, 2, 4, 2, 64, 0, 1)
    assert ws2 == lib.estp_attn_importance_workspace_size(100, 2, 60, 2, 4, 2, 64, 0)
    assert ws1 == lib.estp_attn_importance_from_lse_workspace_size(100, 2, 60, 2, 4, 2, 64, 0)
    w2 = (ctypes.c_float * 2)(1.0, 0.5)
    base = [FAKE, FAKE, None, FAKE, 2, 60, 100, 2, 4, 2, 64, 0.125, w2, 1, 0, FAKE, WS, ws2, None]

    def call(**kw):
        a = list(base)
        idx = {"Q": 0, "lse": 2, "B": 4, "L": 7, "dh": 10, "lw": 12, "flags": 13, "wsb": 17}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.estp_attn_importance_ex(*a)

    assert call(Q=None) == 1
    assert call(B=0) == 1
    assert call(flags=4) == 1
    assert call(lw=(ctypes.c_float * 2)(1.0, float("nan"))) == 1
    assert call(dh=96) == 2
    assert call(L=65, lw=(ctypes.c_float * 65)(*([1.0] * 65))) == 2  # more weighted layers than supported
    assert call(wsb=ws2 - 1) == 3
    assert call(lse=FAKE, wsb=ws1 - 1) == 3


@needs_no_gpu
def test_analysis_validation():
    lib = estp.load()
    assert lib.estp_misalignment(None, FAKE, FAKE, 2, 0.4, 0.4, FAKE, None) == 1
    assert lib.estp_misalignment(FAKE, FAKE, FAKE, 0, 0.4, 0.4, FAKE, None) == 1
    assert lib.estp_misalignment(FAKE, FAKE, FAKE, 2, 1.5, 0.4, FAKE, None) == 1
    assert lib.estp_sjf_padding(None, None, 4, 2, FAKE, None) == 1
    assert lib.estp_sjf_padding(FAKE, None, 4, 0, FAKE, None) == 1


@needs_no_gpu
def test_launch_size_limits():
    # shapes whose grids would pass 2^32 work-items are refused before any device work
    lib = estp.load()
    n = 300_000_000  # bf16 entropy: 16 slices x ceil(n / 256) workgroups of 256 threads
    ws = lib.estp_token_entropy_workspace_size(n, 32, 4096, 0)
    assert lib.estp_token_entropy(FAKE, FAKE, n, 32, 4096, 0, FAKE, None, WS, ws, None) == 2
    assert b"launch" in lib.estp_last_error()
    n = 2_000_000_000  # importance: 2 x (n / 256) x L x Hq fp32 pass-1 workgroups
    ws = lib.estp_attn_importance_workspace_size(n, 1, n, 1, 2, 2, 64, 0)
    assert lib.estp_attn_importance(FAKE, FAKE, FAKE, 1, n, n, 1, 2, 2, 64, 0.125, 0, FAKE, WS, ws, None) == 2
    assert b"launch" in lib.estp_last_error()
    B, T, d = (1 << 20) - 1, 2048, 8192  # pooling: B x d / 512 one-kernel workgroups of 512 threads
    ws = lib.estp_combine_pool_workspace_size(B * T, B, T, d, 0)
    args = [FAKE, FAKE, FAKE, FAKE, B, T, B * T, d, 0.5, 0.5, 1.0, 0, 0, FAKE, None, None, WS, ws, None]
    assert lib.estp_combine_pool(*args) == 2
    assert b"launch" in lib.estp_last_error()
