"""Seeded synthetic inputs of the draft side of a decoding step.

The paper pairs each target with its released EAGLE-3 draft model (Appendix A); those
checkpoints are not used here. The stand-in draft head has the EAGLE-3 shape for an 8B Llama
target: hidden size 4096 and a reduced draft vocabulary of 32000 ids mapped into the
128256-id target vocabulary. Draft LM-head weights are bf16 ~N(0, 0.02), draft hidden states
bf16 ~N(0, 1), one fresh [4B, H] block per draft step (four frontier slots per request), and
the id map is a seeded sorted subset of the target vocabulary. Tree shapes (nsteps, topk, ndt)
are drawn from the ends and midpoints of the paper's range (3,4,4) <-> (7,1,8).

Like ``synth``, this module only draws random numbers and lays them out.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .synth import BASE_SEED, bf16_normal, bf16_weights

_S_DHIDDEN, _S_DMAP, _S_DSHAPE, _S_DROOT = 5, 6, 7, 8
DRAFT_WEIGHT_TAG = 1     # draft LM-head weights use their own key stream

# Shapes in the paper's range, wide-shallow end first.
DRAFT_SHAPES = ((3, 4, 4), (4, 3, 5), (5, 2, 6), (6, 2, 7), (7, 1, 8))

DRAFT_CONFIGS = {
    "llama31_8b_draft_b1": dict(H=4096, V=32000, V_target=128256, B=1),
    "llama31_8b_draft_b32": dict(H=4096, V=32000, V_target=128256, B=32),
}

TOPK_SLOTS = 4           # draft rows per request (frontier slots)


def draft_weights(V: int, H: int) -> np.ndarray:
    """Draft LM-head weight [V, H] as raw bf16 bits (cached, read-only)."""
    return bf16_weights(V, H, 0.02, DRAFT_WEIGHT_TAG)


def draft_hidden(B: int, H: int, step: int, seed: int = 0) -> np.ndarray:
    """Draft hidden states [4B, H] (raw bf16 bits) of one draft step."""
    rng = np.random.default_rng([BASE_SEED, _S_DHIDDEN, B, H, step, seed])
    return bf16_normal(rng, (TOPK_SLOTS * B, H), 1.0)


def draft_vocab_map(V: int, V_target: int) -> np.ndarray:
    """Sorted distinct target ids for the V draft ids (int32)."""
    rng = np.random.default_rng([BASE_SEED, _S_DMAP, V, V_target])
    return np.sort(rng.choice(V_target, size=V, replace=False)).astype(np.int32)


def draft_shapes(B: int, seed: int = 0) -> np.ndarray:
    """A (nsteps, topk, ndt) per request, [B, 3] int32."""
    rng = np.random.default_rng([BASE_SEED, _S_DSHAPE, B, seed])
    return np.array([DRAFT_SHAPES[i] for i in rng.integers(0, len(DRAFT_SHAPES), B)],
                    dtype=np.int32).reshape(B, 3)


def root_tokens(B: int, V_target: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng([BASE_SEED, _S_DROOT, B, V_target, seed])
    return rng.integers(0, V_target, B).astype(np.int32)


@dataclass
class DraftWorkload:
    name: str
    H: int
    V: int
    V_target: int
    B: int

    def weights(self) -> np.ndarray:
        return draft_weights(self.V, self.H)

    def hidden(self, step: int, seed: int = 0) -> np.ndarray:
        return draft_hidden(self.B, self.H, step, seed)

    def vocab_map(self) -> np.ndarray:
        return draft_vocab_map(self.V, self.V_target)


def make_draft_workload(name: str) -> DraftWorkload:
    c = DRAFT_CONFIGS[name]
    return DraftWorkload(name=name, **c)
