"""fp64 CPU oracle of the ESTP scoring and pooling path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it, to check and to time the HIP
library against plain, slow definitions.  It shares no code with the HIP path.

Every function takes bf16 bit patterns (uint16) or float arrays, widens them
exactly to float64 and evaluates the paper's definitions:

* ``token_entropy``      - Eq. 2 (Section 4.2); ``vocab_argmax`` - the mode of
  the same next-token distribution (largest logit, lowest index among ties)
* ``attn_importance``    - Eq. 1 (Section 4.1); ``attn_importance_tail``
  gives the same S_j for the last m keys of one prompt from its last m rows,
  ``attn_importance_keys`` for any set of keys of one prompt from the rows
  that reach them;
  ``attn_row_lse`` is the log normaliser of every attention row and
  ``attn_importance_from_lse`` forms S_j from given row normalisers
* ``combine_weights``    - Eq. 3 and Eq. 4 (Section 4.2)
* ``pool``               - Eq. 5 (Section 4.2)
* ``predict``            - the MLP length head with Eq. 7 (Section 4.3)
* ``soft_labels``, ``length_loss`` - Eq. 6 and Eq. 8 (Section 4.3)
* ``length_bin``, ``head_loss_and_grads``, ``adamw_step``, ``head_train_step`` - one
  training step of the K-bin head: Eq. 8 loss, its gradients, AdamW (Section 5.1)
* ``misalignment_counts`` - the entropy / semantics percentile split (Fig. 1b, Section 1)
* ``sjf_padding``        - padding and completion time of static SJF batches (Section 5.4)

``oracle.bruteforce`` re-derives the same quantities with pure-Python loops
for tiny shapes; the tests pin this module against it, against closed forms
and against invariants the definitions fix.
"""
from .estp_oracle import (  # noqa: F401
    widen,
    token_entropy,
    vocab_argmax,
    attn_importance,
    attn_importance_tail,
    attn_importance_keys,
    attn_row_lse,
    attn_importance_from_lse,
    combine_weights,
    pool,
    predict,
    soft_labels,
    length_loss,
    length_bin,
    head_loss_and_grads,
    adamw_step,
    head_train_step,
    misalignment_counts,
    sjf_padding,
    run_path,
)
