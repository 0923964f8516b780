"""Plain fp64 CPU oracle for the fused attention-distillation KL primitive.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package. The product path (the HIP library and its Python binding) never
imports it, and this package imports nothing from the product path: the two
share no code. Inputs are plain NumPy arrays produced by the seeded generator
in ``paper_2606_20005_amd.inputs``, which holds none of the method's
arithmetic.

Modules
-------
kl_oracle     the plain definition (Sec. 2.1, eq:kl-def / eq:kl-case1 /
              eq:kl-case2): explicit P1 and P2 row block by row block in fp64.
sigmoid_oracle  the same divergence under sigmoid attention scores with no
              normalisation (Sec. 3.1, "Generalizability beyond Softmax"): the
              generalized KL of the two score rows and its gradients.
online_model  the online forward (Sec. 3.2) evaluated from per-tile partial
              states folded with the split-K merge of Sec. 3.3, in fp64. It
              is not the oracle; it pins the paper's online derivation
              (eq:kl-final, eq:acc-invariant) to the plain definition so that
              a GPU/oracle mismatch can be attributed.
"""
from .kl_oracle import (  # noqa: F401
    forward,
    backward,
    forward_rows,
    logit_grads_rows,
    dq_rows,
    dk_rows,
    head_stats_all_rows,
    allowed_mask,
)
from .online_model import online_forward_head, split_merge_forward_head  # noqa: F401
from . import sigmoid_oracle  # noqa: F401,E402
