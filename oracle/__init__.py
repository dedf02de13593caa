"""Oracle for the ZeroLock chunk-local update -- TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 NumPy implementation of what one chunk's update computes
(Sec. II.A, Eq. (1)-(6), the KL form of the local loss in Sec. II.C, the
static-head readout of Sec. III-B, gradient accumulation over an update
window and on-device AdamW of Sec. III).  It shares no code with the HIP
path and must only be imported by tests, the package's smoke check and the
benchmark's CPU-baseline leg.  Nothing in the product path may call it.

Pins (see tests/test_oracle_*.py): finite differences of every gradient,
closed forms (uniform head, identity chunk, AdamW first step), torch-CPU
library routines in fp64 (sdpa, norms, activations, cross-entropy, KL,
torch.optim.AdamW/SGD), the Lemma 2/3 identities of Sec. II.C, and the
coincidence of the single-chunk local update with ordinary backpropagation.
Parity unpinned: which KL direction the paper's own runs used (both are
implemented and pinned internally), and the paper's unstated alpha.
"""
from .chunk import (  # noqa: F401
    OracleConfig,
    chunk_forward_ref,
    chunk_update_ref,
    chunk_grads_ref,
    global_bp_ref,
    bf16_round,
)
from .objective import local_objective_ref, head_logits_ref  # noqa: F401
from .optim import adamw_step_ref, sgd_step_ref  # noqa: F401
