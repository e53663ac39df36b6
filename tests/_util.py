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
