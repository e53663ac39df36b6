"""Seeded, block-addressable synthetic inputs.

Every tensor is drawn in blocks of ``ROW_BLOCK`` rows; block ``k`` of tensor
``tid`` uses its own PCG64 stream seeded by ``SeedSequence([seed, tid, k])``.
That makes generation reproducible, parallel (NumPy releases the GIL while it
fills arrays) and random-access: the oracle can regenerate just the rows it
samples from a full-size workload without drawing the rest.

Value recipe (per workload, see ``synth.workloads``):

* hidden states: each row ~ N(0, 1) per element, divided by its own RMS
  (so every row has RMS 1); in workloads with outliers, exactly
  ``round(outlier_frac * T_b)`` tokens of each prompt, chosen by a seeded
  permutation, are multiplied by 4;
* LM-head weight ``W[V, d]`` ~ N(0, 0.02);
* post-RoPE queries and keys ~ N(0, 1); with ``q_head_scale`` the queries of
  (layer, head) are multiplied by ``s ~ U(0.5, 2)`` to vary attention
  sharpness (the kernel's own score scale stays 1/sqrt(dh));
* ragged prompt lengths ``round(exp(U(ln 32, ln 4096)))`` clipped to range;
* length head ``W1[Hdn, d]``, ``W2[K, Hdn]`` ~ N(0, 0.02), biases 0,
  bin centres (K > 1) evenly spaced.

bfloat16 values are produced by round-to-nearest-even from float32 and kept
as ``uint16`` bit patterns, the exact bytes both paths consume.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence

import numpy as np

from .workloads import Workload

ROW_BLOCK = 256
DEFAULT_SEED = 42

# tensor ids for the per-block seed sequences
_T_LENGTHS = 1
_T_HIDDEN = 2
_T_OUTLIER = 3
_T_LMHEAD = 4
_T_QSCALE = 5
_T_Q = 6
_T_K = 7
_T_W1 = 8
_T_W2 = 10


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# ----------------------------------------------------------------------------- bf16 bits

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even); return uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _finish(x32: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(x32) if dtype == "bf16" else np.ascontiguousarray(x32, dtype=np.float32)


# ----------------------------------------------------------------------------- lengths

def prompt_lengths(w: Workload, seed: int = DEFAULT_SEED) -> np.ndarray:
    if w.seq_len is not None:
        return np.full(w.n_prompts, w.seq_len, dtype=np.int64)
    g = _rng(seed, _T_LENGTHS)
    u = g.uniform(np.log(w.ragged_min), np.log(w.ragged_max), size=w.n_prompts)
    return np.clip(np.rint(np.exp(u)), w.ragged_min, w.ragged_max).astype(np.int64)


def cu_seqlens_from_lengths(lengths: Sequence[int]) -> np.ndarray:
    lengths = np.asarray(lengths, dtype=np.int64)
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    return cu.astype(np.int32)


# ----------------------------------------------------------------------------- row tensors

def _block_rows(rows: Optional[np.ndarray], n_rows: int):
    """Yield (block index, global rows in block wanted, positions in output)."""
    if rows is None:
        nb = (n_rows + ROW_BLOCK - 1) // ROW_BLOCK
        for k in range(nb):
            lo, hi = k * ROW_BLOCK, min(n_rows, (k + 1) * ROW_BLOCK)
            yield k, None, slice(lo, hi)
    else:
        rows = np.asarray(rows, dtype=np.int64)
        if rows.size and (rows.min() < 0 or rows.max() >= n_rows):
            raise IndexError("row index out of range")
        blocks = rows // ROW_BLOCK
        for k in np.unique(blocks):
            pos = np.nonzero(blocks == k)[0]
            yield int(k), rows[pos] - k * ROW_BLOCK, pos


def _gen_rows(n_rows: int, width: int, rows: Optional[np.ndarray], dtype: str, block_fn) -> np.ndarray:
    """Fill an [n_out, width] array block by block; ``block_fn(k, nrows)`` -> float32 [nrows, width]."""
    n_out = n_rows if rows is None else len(rows)
    out = np.empty((n_out, width), dtype=np.uint16 if dtype == "bf16" else np.float32)

    def work(item):
        k, local, pos = item
        nrows = min(ROW_BLOCK, n_rows - k * ROW_BLOCK)
        blk = block_fn(k, nrows)
        if local is not None:
            blk = blk[local]
        out[pos] = _finish(blk, dtype)

    items = list(_block_rows(rows, n_rows))
    if len(items) <= 2:
        for it in items:
            work(it)
    else:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(work, items))
    return out


def _outlier_tokens(w: Workload, seed: int, lengths: np.ndarray) -> np.ndarray:
    """Global indices of the outlier tokens (exactly round(frac * T_b) per prompt)."""
    if w.outlier_frac <= 0:
        return np.zeros(0, dtype=np.int64)
    cu = cu_seqlens_from_lengths(lengths).astype(np.int64)
    idx = []
    for b, T in enumerate(lengths):
        n = int(round(w.outlier_frac * int(T)))
        if n == 0:
            continue
        g = _rng(seed, _T_OUTLIER, b)
        idx.append(cu[b] + np.sort(g.permutation(int(T))[:n]))
    return np.concatenate(idx) if idx else np.zeros(0, dtype=np.int64)


def hidden_rows(w: Workload, seed: int = DEFAULT_SEED, lengths: Optional[np.ndarray] = None,
                rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Hidden states X [n_tok, d] (or the given global rows): bf16 bits or float32."""
    if lengths is None:
        lengths = prompt_lengths(w, seed)
    n_tok = int(np.sum(lengths))
    outl = np.zeros(n_tok, dtype=bool)
    outl[_outlier_tokens(w, seed, lengths)] = True

    def block(k, nrows):
        g = _rng(seed, _T_HIDDEN, k)
        z = g.standard_normal((nrows, w.d), dtype=np.float32)
        rms = np.sqrt(np.mean(np.square(z, dtype=np.float32), axis=1, dtype=np.float32), dtype=np.float32)
        z /= rms[:, None]
        m = outl[k * ROW_BLOCK: k * ROW_BLOCK + nrows]
        if m.any():
            z[m] *= np.float32(4.0)
        return z

    return _gen_rows(n_tok, w.d, rows, w.dtype, block)


def lm_head_rows(w: Workload, seed: int = DEFAULT_SEED, rows: Optional[np.ndarray] = None) -> np.ndarray:
    """LM-head weight W [V, d] (nn.Linear layout), entries N(0, 0.02)."""
    def block(k, nrows):
        g = _rng(seed, _T_LMHEAD, k)
        z = g.standard_normal((nrows, w.d), dtype=np.float32)
        z *= np.float32(0.02)
        return z

    return _gen_rows(w.V, w.d, rows, w.dtype, block)


def query_head_scales(w: Workload, seed: int = DEFAULT_SEED) -> np.ndarray:
    """Per (layer, query head) multiplier of the queries: U(0.5, 2) or all ones."""
    if not w.q_head_scale:
        return np.ones((w.L, w.Hq), dtype=np.float32)
    g = _rng(seed, _T_QSCALE)
    return g.uniform(0.5, 2.0, size=(w.L, w.Hq)).astype(np.float32)


def qk_layer(w: Workload, which: str, layer: int, seed: int = DEFAULT_SEED,
             lengths: Optional[np.ndarray] = None, rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Post-RoPE queries [n_tok, Hq, dh] or keys [n_tok, Hkv, dh] of one layer."""
    if lengths is None:
        lengths = prompt_lengths(w, seed)
    n_tok = int(np.sum(lengths))
    H = w.Hq if which == "q" else w.Hkv
    tid = _T_Q if which == "q" else _T_K
    scales = query_head_scales(w, seed)[layer] if which == "q" else None

    def block(k, nrows):
        g = _rng(seed, tid, layer, k)
        z = g.standard_normal((nrows, H * w.dh), dtype=np.float32)
        if scales is not None:
            z = (z.reshape(nrows, H, w.dh) * scales[None, :, None]).reshape(nrows, H * w.dh)
        return z

    out = _gen_rows(n_tok, H * w.dh, rows, w.dtype, block)
    return out.reshape(out.shape[0], H, w.dh)


def mlp_head(w: Workload, seed: int = DEFAULT_SEED, n_bins: Optional[int] = None):
    """Length head: W1 [Hdn, d], b1 [Hdn], W2 [K, Hdn], b2 [K], centres [K] (float32)."""
    Hdn, K = w.head
    if n_bins is not None:
        K = n_bins
    W1 = (_rng(seed, _T_W1).standard_normal((Hdn, w.d), dtype=np.float32) * np.float32(0.02))
    W2 = (_rng(seed, _T_W2).standard_normal((K, Hdn), dtype=np.float32) * np.float32(0.02))
    b1 = np.zeros(Hdn, dtype=np.float32)
    b2 = np.zeros(K, dtype=np.float32)
    # evenly spaced bin centres over output lengths 0..4096 tokens (used only when K > 1)
    centres = ((np.arange(K, dtype=np.float32) + np.float32(0.5)) * np.float32(4096.0 / K)).astype(np.float32)
    return W1, b1, W2, b2, centres


# ----------------------------------------------------------------------------- bundle

def make_inputs(w: Workload, seed: int = DEFAULT_SEED, parts: Sequence[str] = ("X", "W", "Q", "K", "head")):
    """Draw every input of the path for workload ``w``.

    Returns a dict with ``lengths``, ``cu_seqlens`` (int32 [B+1]) and, as
    requested, ``X`` [n_tok, d], ``W`` [V, d], ``Q`` [L, n_tok, Hq, dh],
    ``K`` [L, n_tok, Hkv, dh] (bf16 bits as uint16, or float32), and the
    length head ``W1, b1, W2, b2, centres``.
    """
    lengths = prompt_lengths(w, seed)
    cu = cu_seqlens_from_lengths(lengths)
    n_tok = int(cu[-1])
    out = {"workload": w, "seed": seed, "lengths": lengths, "cu_seqlens": cu, "n_tok": n_tok}
    if "X" in parts:
        out["X"] = hidden_rows(w, seed, lengths)
    if "W" in parts:
        out["W"] = lm_head_rows(w, seed)
    if "Q" in parts:
        out["Q"] = np.stack([qk_layer(w, "q", l, seed, lengths) for l in range(w.L)])
    if "K" in parts:
        out["K"] = np.stack([qk_layer(w, "k", l, seed, lengths) for l in range(w.L)])
    if "head" in parts:
        out["W1"], out["b1"], out["W2"], out["b2"], out["centres"] = mlp_head(w, seed)
    return out
