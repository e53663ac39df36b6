"""Seeded synthetic inputs for the ESTP scoring and pooling path.

This package is shared by the tests, ``bench.py`` and the smoke check: it draws
hidden states, LM-head weights, post-RoPE queries/keys, prompt lengths and the
length-head weights, and rounds them to bfloat16.  It holds none of the
method's arithmetic (no entropy, attention, softmax or pooling): both the HIP
path and the fp64 oracle consume the exact bytes it produces.
"""
from .workloads import WORKLOADS, Workload, get_workload  # noqa: F401
from .inputs import (  # noqa: F401
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_inputs,
    prompt_lengths,
    cu_seqlens_from_lengths,
    hidden_rows,
    lm_head_rows,
    qk_layer,
    mlp_head,
    query_head_scales,
)
