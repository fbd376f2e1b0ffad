"""CPU oracle for the AdaptiveSpec verification path. TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 implementation of what the verification path computes, written from the
paper ("Margins, Not Windows: Training-Free Per-Step Lossy Speculative Decoding"): the target
LM-head logits of every draft-tree row, the per-row max / argmax / log-sum-exp, the margin rule
of Sec. 3.2 Eq. (1), the tree walk that promotes mismatches, the draft top-1 confidence of
Sec. 3.3 Eq. (2), the rolling acceptance history of Sec. 3.3 and the tree shape the Draft
Confidence Score selects (Sec. 3.3, Eq. (2)). ``tree_oracle`` covers the steps on either side:
the draft-side top-k and the growth and pruning of the draft tree (Sec. 2, "Draft"), the tree
attention metadata of the target forward and the commit of the accepted path.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. It shares no code with the HIP path (``paper_2609_02897_amd``); both read inputs from
``workloads`` only.

Parity pins live in ``tests/oracle_pins.py`` and ``tests/tree_pins.py``. Every function has a pin. Where the paper does
not fix a result (the walk's sibling choice, the promotion count, the acceptance observation,
the history reset on a breaker trip, the rounding of the tree shape and the starting
configuration), the docstring names the reading taken, and the pins check the code against
that reading stated independently.
"""

from .asv_oracle import (  # noqa: F401
    LN_BAND,
    Params,
    ReqState,
    accept_flags,
    draft_confidence,
    logits,
    row_stats,
    row_top8,
    state_init,
    state_update,
    tree_shape,
    tree_shape_slack,
    verify,
    walk,
    walk_bands,
    widen_bf16,
    widen_weights,
)
from .tree_oracle import (  # noqa: F401
    DraftTree,
    commit,
    draft_top1_prob,
    draft_topk,
    draft_tree_init,
    draft_tree_prune,
    draft_tree_step,
    draft_trees_to_batch,
    tree_meta,
)
