"""Seeded synthetic inputs shaped like the paper's verification workloads.

The paper evaluates on Llama-3.1-8B, DeepSeek-R1-Distill-Llama-8B and Qwen3-8B with EAGLE-3
draft trees (Section 4.1, Appendix A); its datasets and checkpoints are not used here. These
seeded inputs stand in for them: target LM-head shapes H=4096 with V=128256 (Llama-3.1 vocab)
or V=151936 (Qwen3 vocab), bf16 weights ~N(0, 0.02), bf16 hidden states ~N(0, 1), and draft
trees in the EAGLE-3 regime (a root for the last committed token plus drafted nodes, parent
index < child index, requests packed contiguously).

Drafted tokens are described by random *choices* drawn here ("the target's top-1", "a uniform
pick among the target's top-8", "a uniform vocabulary id"). Turning a choice into a token id
needs the target's top-8 for the parent row, which only a logits computation can give; that
table is passed in by the caller (:func:`resolve_drafts`), so this module never computes a
logit.

Every array is derived from ``numpy.random.default_rng([BASE_SEED, ...])`` keys and is
identical on every machine with the same numpy.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from functools import lru_cache
from typing import Callable, Optional, Sequence

import numpy as np

BASE_SEED = 260902897

# Stream tags of the seed keys.
_S_WEIGHT, _S_HIDDEN, _S_TREE, _S_DRAFT, _S_DLOGIT = 0, 1, 2, 3, 4

# Rows of W generated per independent key; fixed so the matrix never depends on thread count.
_W_CHUNK_ROWS = 2048


def _mix_const(p_arg: float, p_top8: float) -> Callable[[int], tuple]:
    return lambda depth: (p_arg, p_top8)


def _mix_decay(depth: int) -> tuple:
    # argmax probability 0.5 at depth 1, decaying by 0.8 per level; the rest split 3:2
    # between a top-8 pick and a uniform vocabulary id.
    p_arg = 0.5 * 0.8 ** (depth - 1)
    rest = 1.0 - p_arg
    return (p_arg, 0.6 * rest)


# The five synthetic configurations. ``trees`` names a builder in build_tree.
CONFIGS = {
    0: dict(name="tiny_h256_v4096_n8", H=256, V=4096, B=1, trees="tiny", taus=(0.3,),
            mix=_mix_const(0.5, 0.3), steps=1, draft_logits=False),
    1: dict(name="llama31_8b_b1_n60", H=4096, V=128256, B=1, trees="eagle60",
            taus=(0.1, 0.3), mix=_mix_decay, steps=1, draft_logits=False),
    2: dict(name="qwen3_8b_b8_adaptive", H=4096, V=151936, B=8, trees="adaptive",
            taus=(0.2,), mix=_mix_const(0.5, 0.3), steps=32, draft_logits=True),
    3: dict(name="llama31_8b_b32x64", H=4096, V=128256, B=32, trees="level8x8",
            taus=(0.3,), mix=_mix_const(0.6, 0.25), steps=1, draft_logits=False),
    4: dict(name="qwen3_8b_b64_sweep", H=4096, V=151936, B=64, trees="chain_or_wide",
            taus=(0.05, 0.1, 0.3, 1.0), mix=_mix_const(0.5, 0.3), steps=1,
            draft_logits=False),
}


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); raw uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Raw bf16 bits to float32 (exact). Used for input statistics only."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    x *= np.float32(std)
    return round_to_bf16_bits(x)


def _w_chunk(args):
    V, H, std, tag, c = args
    r0 = c * _W_CHUNK_ROWS
    rows = min(_W_CHUNK_ROWS, V - r0)
    rng = np.random.default_rng([BASE_SEED, _S_WEIGHT, tag, V, H, c])
    return bf16_normal(rng, (rows, H), std)


@lru_cache(maxsize=2)
def bf16_weights(V: int, H: int, std: float = 0.02, tag: int = 0) -> np.ndarray:
    """LM-head weight W[V, H] as raw bf16 bits, ~N(0, std) before rounding.

    Generated in fixed 2048-row chunks, each from its own key, on a thread pool. The same
    (V, H, std, tag) gives the same matrix whatever the thread count. The result is cached
    (read-only) because the 8B-shaped matrices take seconds to draw.
    """
    nchunks = (V + _W_CHUNK_ROWS - 1) // _W_CHUNK_ROWS
    out = np.empty((V, H), dtype=np.uint16)
    workers = max(1, min(16, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        for c, blk in enumerate(ex.map(_w_chunk, [(V, H, std, tag, c) for c in range(nchunks)])):
            out[c * _W_CHUNK_ROWS: c * _W_CHUNK_ROWS + blk.shape[0]] = blk
    out.flags.writeable = False
    return out


def _dl_chunk(args):
    key, V, r0, rows = args
    x = np.random.default_rng([BASE_SEED, _S_DLOGIT, *key, r0]).standard_normal(
        (rows, V), dtype=np.float32)
    x *= np.float32(2.0)
    return x


def draft_logit_matrix(key, N: int, V: int, rows_per_chunk: int = 32) -> np.ndarray:
    """Draft-model logits [N, V] float32 ~N(0, 2), in fixed row chunks with their own keys
    (drawn on a thread pool; independent of the thread count)."""
    out = np.empty((N, V), dtype=np.float32)
    jobs = [(tuple(key), V, r0, min(rows_per_chunk, N - r0)) for r0 in range(0, N, rows_per_chunk)]
    workers = max(1, min(16, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        for (_, _, r0, rows), blk in zip(jobs, ex.map(_dl_chunk, jobs)):
            out[r0:r0 + rows] = blk
    return out


# ----------------------------------------------------------------------------- trees

def tree_depths(parent: np.ndarray) -> np.ndarray:
    """Depth of every node of one tree (root = 0); parent[c] < c is assumed."""
    d = np.zeros(len(parent), dtype=np.int32)
    for c in range(1, len(parent)):
        d[c] = d[parent[c]] + 1
    return d


def _bfs_renumber(parent: Sequence[int]) -> np.ndarray:
    """Renumber a tree (parent[c] < c) so levels are contiguous, keeping order inside a level."""
    parent = np.asarray(parent, dtype=np.int64)
    depth = tree_depths(parent)
    order = np.lexsort((np.arange(len(parent)), depth))   # by depth, then old id
    new_id = np.empty_like(order)
    new_id[order] = np.arange(len(order))
    out = np.full(len(parent), -1, dtype=np.int32)
    for old in range(1, len(parent)):
        out[new_id[old]] = new_id[parent[old]]
    return out


def _tree_tiny(rng):
    # 8 nodes, depth <= 4, branching <= 3, each new node under a uniformly chosen open node.
    parent, depth, kids = [-1], [0], [0]
    for _ in range(7):
        open_nodes = [i for i in range(len(parent)) if depth[i] < 4 and kids[i] < 3]
        p = int(open_nodes[rng.integers(len(open_nodes))])
        parent.append(p)
        depth.append(depth[p] + 1)
        kids.append(0)
        kids[p] += 1
    return _bfs_renumber(parent)


def _tree_levels(rng, levels):
    # Root plus fixed level sizes; each node's parent is uniform over the previous level.
    parent = [-1]
    prev = [0]
    for size in levels:
        cur = []
        for _ in range(size):
            parent.append(int(prev[rng.integers(len(prev))]))
            cur.append(len(parent) - 1)
        prev = cur
    return np.asarray(parent, dtype=np.int32)


def _tree_chain_plus(rng, n, D):
    # A chain of depth D, then the remaining nodes attached uniformly to nodes of depth < D.
    parent = [-1] + list(range(D))
    depth = list(range(D + 1))
    while len(parent) < n:
        cand = [i for i in range(len(parent)) if depth[i] < D]
        p = int(cand[rng.integers(len(cand))])
        parent.append(p)
        depth.append(depth[p] + 1)
    return _bfs_renumber(parent)


def _tree_wide(rng, n):
    # 32 children of the root, then n - 33 level-2 nodes under uniform level-1 parents.
    parent = [-1] + [0] * 32
    for _ in range(n - 33):
        parent.append(int(1 + rng.integers(32)))
    return _bfs_renumber(parent)


def build_tree(kind: str, rng: np.random.Generator, b: int) -> np.ndarray:
    """Parent array (local ids, root first) of request ``b`` for a named tree family."""
    if kind == "tiny":
        return _tree_tiny(rng)
    if kind == "eagle60":
        return _tree_levels(rng, [10, 10, 10, 10, 10, 9])
    if kind == "level8x8":
        return _tree_levels(rng, [8, 8, 8, 8, 8, 8, 8, 7])
    if kind == "adaptive":
        n = int(rng.integers(8, 97))
        D = min(int(rng.integers(2, 11)), n - 1)
        return _tree_chain_plus(rng, n, D)
    if kind == "chain_or_wide":
        if b % 2 == 0:
            return np.asarray([-1] + list(range(16)), dtype=np.int32)
        return _tree_wide(rng, int(rng.integers(34, 129)))
    raise ValueError(f"unknown tree family {kind!r}")


# ----------------------------------------------------------------------------- drafts

def draft_choices(rng: np.random.Generator, depth: np.ndarray, V: int,
                  mix: Callable[[int], tuple]):
    """Per node: kind (0 target top-1, 1 uniform pick in the target top-8, 2 uniform id),
    the top-8 rank for kind 1 and the vocabulary id for kind 2. Root entries are -1."""
    n = len(depth)
    u = rng.random(n)
    rank = rng.integers(0, 8, size=n).astype(np.int32)
    uid = rng.integers(0, V, size=n).astype(np.int32)
    kind = np.full(n, -1, dtype=np.int8)
    for i in range(n):
        if depth[i] == 0:
            continue
        p_arg, p_top8 = mix(int(depth[i]))
        kind[i] = 0 if u[i] < p_arg else (1 if u[i] < p_arg + p_top8 else 2)
    rank[depth == 0] = -1
    uid[depth == 0] = -1
    return kind, rank, uid


def resolve_drafts(kind: np.ndarray, rank: np.ndarray, uid: np.ndarray,
                   parent: np.ndarray, top8: np.ndarray) -> np.ndarray:
    """Drafted token of every node from its choice and the target's top-8 of its parent row.

    ``top8[r]`` lists row r's eight highest-logit vocabulary ids, best first (supplied by the
    caller). Roots get -1.
    """
    tok = np.full(len(kind), -1, dtype=np.int32)
    for c in range(len(kind)):
        if kind[c] < 0:
            continue
        p = parent[c]
        if kind[c] == 0:
            tok[c] = top8[p, 0]
        elif kind[c] == 1:
            tok[c] = top8[p, rank[c]]
        else:
            tok[c] = uid[c]
    return tok


# ----------------------------------------------------------------------------- workloads

@dataclass
class Workload:
    """One verify call's inputs (host numpy arrays). Global node ids index ``hidden`` rows."""
    name: str
    H: int
    V: int
    B: int
    N: int
    req_offsets: np.ndarray          # int32 [B+1]
    parent: np.ndarray               # int32 [N], global ids, -1 at roots
    depth: np.ndarray                # int32 [N]
    tau: np.ndarray                  # float32 [B]
    hidden: np.ndarray               # uint16 [N, H] bf16 bits
    kind: np.ndarray                 # int8 [N]
    rank: np.ndarray                 # int32 [N]
    uid: np.ndarray                  # int32 [N]
    draft_logits: Optional[np.ndarray] = None   # float32 [N, V] or None
    w_std: float = 0.02
    w_tag: int = 0
    draft_tok: Optional[np.ndarray] = field(default=None)  # int32 [N] once resolved

    def weights(self) -> np.ndarray:
        return bf16_weights(self.V, self.H, self.w_std, self.w_tag)

    def with_drafts(self, top8: np.ndarray) -> "Workload":
        self.draft_tok = resolve_drafts(self.kind, self.rank, self.uid, self.parent, top8)
        return self


def _pack(trees):
    sizes = [len(t) for t in trees]
    off = np.zeros(len(trees) + 1, dtype=np.int32)
    off[1:] = np.cumsum(sizes)
    parent = np.empty(off[-1], dtype=np.int32)
    depth = np.empty(off[-1], dtype=np.int32)
    for b, t in enumerate(trees):
        t = np.asarray(t, dtype=np.int32)
        g = np.where(t >= 0, t + off[b], -1)
        parent[off[b]:off[b + 1]] = g
        depth[off[b]:off[b + 1]] = tree_depths(t)
    return off, parent, depth


def custom_workload(name: str, H: int, V: int, trees, tau, *, seed: int,
                    mix=_mix_const(0.5, 0.3), draft_logits: bool = False,
                    w_std: float = 0.02, w_tag: int = 1, hidden_std: float = 1.0) -> Workload:
    """Workload from explicit local parent arrays (one per request)."""
    off, parent, depth = _pack(trees)
    N, B = int(off[-1]), len(trees)
    hidden = bf16_normal(np.random.default_rng([BASE_SEED, _S_HIDDEN, 1000 + seed]),
                         (N, H), hidden_std)
    kind, rank, uid = draft_choices(np.random.default_rng([BASE_SEED, _S_DRAFT, 1000 + seed]),
                                    depth, V, mix)
    tau = np.broadcast_to(np.asarray(tau, dtype=np.float32), (B,)).copy()
    dl = draft_logit_matrix((1000 + seed,), N, V) if draft_logits else None
    return Workload(name, H, V, B, N, off, parent, depth, tau, hidden, kind, rank, uid, dl,
                    w_std, w_tag)


def make_trees(cfg: int, step: int = 0):
    """The seeded trees of configuration ``cfg`` at decode step ``step`` alone, as
    (req_offsets, parent, depth): the same values make_workload draws, without the hidden
    states and logits."""
    c = CONFIGS[cfg]
    trng = np.random.default_rng([BASE_SEED, cfg, step, _S_TREE])
    return _pack([build_tree(c["trees"], trng, b) for b in range(c["B"])])


def make_workload(cfg: int, step: int = 0, tau: Optional[float] = None) -> Workload:
    """The seeded inputs of synthetic configuration ``cfg`` at decode step ``step``."""
    c = CONFIGS[cfg]
    H, V, B = c["H"], c["V"], c["B"]
    trng = np.random.default_rng([BASE_SEED, cfg, step, _S_TREE])
    trees = [build_tree(c["trees"], trng, b) for b in range(B)]
    off, parent, depth = _pack(trees)
    N = int(off[-1])
    hidden = bf16_normal(np.random.default_rng([BASE_SEED, cfg, step, _S_HIDDEN]), (N, H), 1.0)
    kind, rank, uid = draft_choices(np.random.default_rng([BASE_SEED, cfg, step, _S_DRAFT]),
                                    depth, V, c["mix"])
    t = c["taus"][-1] if tau is None else tau
    taus = np.full(B, t, dtype=np.float32)
    dl = draft_logit_matrix((cfg, step), N, V) if c["draft_logits"] else None
    return Workload(c["name"], H, V, B, N, off, parent, depth, taus, hidden, kind, rank, uid,
                    dl)
