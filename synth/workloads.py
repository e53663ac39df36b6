"""Named workload shapes for the ESTP scoring and pooling path.

Each preset mirrors one of the workload shapes the path is measured on.  The
paper evaluates on Qwen2.5 and Llama3.2 backbones over the ForeLen prompts
(Section 5.1); neither the weights nor the prompts are available, so these
presets are synthetic stand-ins with the backbone-like shapes listed here and
the value distributions drawn in ``synth.inputs``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    n_prompts: int
    # fixed prompt length, or None for the ragged log-uniform mix
    seq_len: Optional[int]
    d: int
    V: int
    Hq: int
    Hkv: int
    dh: int
    L: int
    dtype: str = "bf16"  # "bf16" or "f32" for X, W, Q, K
    q_head_scale: bool = True  # multiply query head h by s_h ~ U(0.5, 2)
    outlier_frac: float = 0.0  # fraction of tokens per prompt whose hidden state is x4
    ragged_min: int = 32
    ragged_max: int = 4096
    head: Tuple[int, int] = (1024, 1)  # (hidden width, number of bins K)
    description: str = field(default="", compare=False)


WORKLOADS = {
    "tiny": Workload(
        name="tiny", n_prompts=1, seq_len=128, d=64, V=1000, Hq=2, Hkv=2, dh=32, L=1,
        dtype="f32", q_head_scale=False, outlier_frac=0.0, head=(32, 1),
        description="1 prompt x 128 tokens, d=64, V=1000, 2/2 heads of 32, 1 layer, fp32",
    ),
    "qwen": Workload(
        name="qwen", n_prompts=16, seq_len=512, d=1536, V=151936, Hq=12, Hkv=2, dh=128, L=1,
        description="Qwen2.5-1.5B-shaped: 16 x 512 tokens, d=1536, V=151936, 12/2 heads of 128, 1 layer, bf16",
    ),
    "llama": Workload(
        name="llama", n_prompts=32, seq_len=2048, d=4096, V=128256, Hq=32, Hkv=8, dh=128, L=4,
        outlier_frac=0.05,
        description=("Llama-3-8B-shaped: 32 x 2048 tokens, d=4096, V=128256, 32/8 heads of 128, "
                     "importance summed over 4 layers, 5% x4-norm outlier tokens, bf16"),
    ),
    "ragged": Workload(
        name="ragged", n_prompts=256, seq_len=None, d=4096, V=128256, Hq=32, Hkv=8, dh=128, L=1,
        outlier_frac=0.05,
        description=("ragged RL batch: 256 prompts, lengths log-uniform in [32, 4096], Llama-3-8B shapes, "
                     "packed varlen, 4096->1024->1 length head, bf16"),
    ),
    "llama1b": Workload(
        name="llama1b", n_prompts=32, seq_len=2048, d=2048, V=128256, Hq=32, Hkv=8, dh=64, L=4,
        outlier_frac=0.05, head=(1024, 16),
        description=("Llama-3.2-1B-shaped: 32 x 2048 tokens, d=2048, V=128256, 32/8 heads of 64, "
                     "importance summed over 4 layers, 5% x4-norm outlier tokens, 16-bin head, bf16"),
    ),
    "long": Workload(
        name="long", n_prompts=2, seq_len=32768, d=4096, V=128256, Hq=32, Hkv=8, dh=128, L=1,
        outlier_frac=0.05,
        description="long context: 2 x 32768 tokens, Llama-3-8B shapes, 1 layer, bf16",
    ),
}


def get_workload(name: str, **overrides) -> Workload:
    """Return a preset, optionally with fields replaced (e.g. a shorter seq_len for tests)."""
    w = WORKLOADS[name]
    if overrides:
        from dataclasses import replace
        w = replace(w, **overrides)
    return w
