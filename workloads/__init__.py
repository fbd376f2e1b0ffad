"""Seeded synthetic workloads for the AdaptiveSpec verification path.

This package is the only code shared by the CPU oracle (``oracle/``) and the HIP path
(``paper_2609_02897_amd``). It draws random numbers and lays them out; it holds none of the
method's arithmetic (no logits, no reductions, no margin rule, no tree walk).
"""

from .synth import (  # noqa: F401
    BASE_SEED,
    CONFIGS,
    Workload,
    bf16_bits_to_f32,
    bf16_normal,
    bf16_weights,
    build_tree,
    custom_workload,
    draft_choices,
    make_trees,
    make_workload,
    resolve_drafts,
    round_to_bf16_bits,
    tree_depths,
)
from .draft import (  # noqa: F401
    DRAFT_CONFIGS,
    DRAFT_SHAPES,
    DraftWorkload,
    draft_hidden,
    draft_shapes,
    draft_vocab_map,
    draft_weights,
    make_draft_workload,
    root_tokens,
)
