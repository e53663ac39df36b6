"""ESTP scoring and pooling on MI355X (gfx950).

Python face of libestp.so: the four calls of the ESTP path (arXiv 2608.15592)

* ``token_entropy``   - Eq. 2, fused LM-head GEMM with streaming entropy (and, optionally,
  each token's most probable next token); ``token_entropy_noalloc`` - the same with the
  library's own scratch, allocating nothing
* ``attn_importance`` - Eq. 1, two-pass causal attention column means
* ``attn_importance_from_lse`` - Eq. 1 from a prefill's per-row log-sum-exps (one pass)
* ``attn_importance_ex`` - Eq. 1 variants: diagonal left out, per-layer weights, optional LSEs
* ``combine_pool``    - Eq. 3-5, temperature softmax of the fused score and weighted pooling
* ``predict``         - length head (Section 4.3, Eq. 7) and shortest-job-first order
* ``head_train_step`` - one Eq. 6-8 / AdamW training step of the K-bin head
* ``misalignment``, ``sjf_padding`` - the Fig. 1b rank split and static SJF batch padding / JCT

plus ``run_path`` chaining them.  All computation runs in the library's HIP
kernels; torch only supplies device memory and the stream.
"""
from ._lib import (  # noqa: F401
    EXPORTS,
    EstpError,
    LIB_PATH,
    attn_importance,
    attn_importance_from_lse,
    attn_importance_ex,
    combine_pool,
    load,
    predict,
    head_param_views,
    head_train_step,
    misalignment,
    sjf_padding,
    token_entropy,
    token_entropy_noalloc,
    token_entropy_workspace_size,
)
from .path import run_path  # noqa: F401
