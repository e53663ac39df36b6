"""Helpers shared by the GPU tests: host <-> device transfer and comparison rules."""
import numpy as np
import torch


def dev(a: np.ndarray) -> torch.Tensor:
    """numpy array -> device tensor; uint16 arrays are bf16 bit patterns."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(a.copy()).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def check_argmax_margin(got: int, values: np.ndarray, delta: float) -> str:
    """Index of a maximum must match exactly when the runner-up is more than `delta` below;
    inside a near-tie group any member is accepted.  Returns 'exact' or 'tie'."""
    v = np.asarray(values, dtype=np.float64)
    best = int(np.argmax(v))
    srt = np.sort(v)
    gap = srt[-1] - srt[-2] if len(v) > 1 else np.inf
    if gap > delta:
        assert got == best, f"argmax {got} != {best} (gap {gap:.3g} > {delta:.3g})"
        return "exact"
    assert v[got] >= srt[-1] - delta, f"argmax {got} not in the near-tie group"
    return "tie"


def check_order_margin(order_gpu: np.ndarray, y_ref: np.ndarray, delta: np.ndarray) -> int:
    """`order_gpu` must be a permutation that sorts the reference values ascending, with
    swaps allowed only between values closer than `delta`; returns the number of near-tie pairs."""
    order_gpu = np.asarray(order_gpu)
    B = len(y_ref)
    assert sorted(order_gpu.tolist()) == list(range(B)), "order is not a permutation"
    ys = np.asarray(y_ref, dtype=np.float64)[order_gpu]
    d = np.broadcast_to(np.asarray(delta, dtype=np.float64), (B,))[order_gpu]
    ties = 0
    for k in range(B - 1):
        if ys[k + 1] < ys[k]:
            assert ys[k] - ys[k + 1] <= max(d[k], d[k + 1]), f"order inverted at {k}: {ys[k]} > {ys[k + 1]}"
            ties += 1
    # where neighbours are well separated, the order must be the oracle's stable order
    ref = np.argsort(y_ref, kind="stable")
    sep = np.all(np.diff(np.sort(y_ref)) > np.max(delta))
    if sep:
        np.testing.assert_array_equal(order_gpu, ref)
    return ties


def logit_error_bound(X, W, rows) -> np.ndarray:
    """Per-row bound on how far a computed fp32 logit can be from the exact one.

    Any order of fp32 summation of d terms is within gamma_d * sum |terms| of the
    exact sum (gamma_d = d u / (1 - d u), u = 2^-24; fp32 products of fp32 inputs
    add one more rounding each, covered by gamma_{d+1}).  Two logits can then be
    swapped only when their exact values are within the sum of their bounds, so the
    margin is twice the row's largest sum |w_vk x_k| over the vocabulary.
    """
    import oracle
    Xa = np.abs(oracle.widen(np.asarray(X)[rows]))
    Wa = np.abs(oracle.widen(W))
    d = Xa.shape[1]
    u = 2.0 ** -24
    gamma = (d + 1) * u / (1 - (d + 1) * u)
    return 2.0 * gamma * (Xa @ Wa.T).max(axis=1)


def check_vocab_argmax(got: np.ndarray, X, W, rows=None) -> dict:
    """The mode of each row's next-token distribution (largest logit, lowest index among
    ties) against the oracle under the margin rule: exact wherever the oracle's gap from
    the largest to the second-largest logit exceeds the fp32 bound of ``logit_error_bound``;
    inside a near tie, any index whose exact logit is within that bound of the largest.
    Returns counts of exact and near-tie rows."""
    import oracle
    X = np.asarray(X)
    rows = np.arange(X.shape[0]) if rows is None else np.asarray(rows)
    ref = oracle.vocab_argmax(X[rows], W)
    z = oracle.widen(X[rows]) @ oracle.widen(W).T
    delta = logit_error_bound(X, W, rows)
    got = np.asarray(got)
    assert got.shape == (len(rows),)
    assert np.all((got >= 0) & (got < z.shape[1])), "argmax index out of range"
    counts = {"exact": 0, "tie": 0}
    for r in range(len(rows)):
        zr = z[r]
        top2 = np.partition(zr, -2)[-2:] if zr.size > 1 else np.array([-np.inf, zr[0]])
        gap = top2[1] - top2[0]
        if gap > delta[r]:
            assert got[r] == ref[r], f"row {rows[r]}: argmax {got[r]} != {ref[r]} (gap {gap:.3g} > {delta[r]:.3g})"
            counts["exact"] += 1
        else:
            assert zr[got[r]] >= zr[ref[r]] - delta[r], f"row {rows[r]}: {got[r]} not in the near-tie group"
            counts["tie"] += 1
    return counts
